"""UltraEP per-microbatch balancing path for MI355X (gfx950).

Thin ctypes binding of ``libultraep.so`` (C ABI in ``include/ultraep.h``).
Every function has the name of the C entry point it calls and only marshals
arguments: torch tensors supply device memory, torch's current HIP stream is
used unless another one is given, and every step runs in the library's HIP
kernels.  Before a call it checks that every tensor is large enough for the
shapes given, so a kernel never runs past a caller's buffer.  A missing library raises immediately; there is no fallback path.

Reference: "UltraEP: Unleash MoE Training and Inference on Rack-Scale Nodes
with Near-Optimal Load Balancing", arXiv 2606.04101 (Algorithm 1, Sec. 5-6).
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
# the in-tree build; ULTRAEP_LIB names another build of the same sources
# (for example a kernel variant under comparison) without replacing it
LIB_PATH = os.environ.get("ULTRAEP_LIB") or os.path.join(_HERE, "libultraep.so")

ULTRAEP_OK = 0
ULTRAEP_EINVAL = -1
ULTRAEP_ENOSPC = -2
ULTRAEP_EDEVICE = -3
ULTRAEP_EDATA = -4


class UltraEPError(RuntimeError):
    def __init__(self, code, where):
        self.code = code
        super().__init__(f"{where}: {ultraep_strerror(code)} ({code})")


class Group(ctypes.Structure):
    """ultraep_group: R ranks, E experts, n_slot redundant slots per rank,
    quota floor u_min, balancing target beta_num / beta_den."""
    _fields_ = [("R", ctypes.c_int32), ("E", ctypes.c_int32),
                ("n_slot", ctypes.c_int32), ("u_min", ctypes.c_int64),
                ("beta_num", ctypes.c_int32), ("beta_den", ctypes.c_int32)]

    def __init__(self, R, E, n_slot, u_min, beta_num=101, beta_den=100):
        super().__init__(R, E, n_slot, u_min, beta_num, beta_den)

    @property
    def n_main(self):
        return self.E // self.R

    @property
    def S(self):
        return self.n_main + self.n_slot

    @property
    def ncol(self):
        return self.E + self.R * self.n_slot


class PlanBuf(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in
                ("slot_expert", "quota", "host_ptr", "host_rank", "host_pslot",
                 "reroute", "stats")]


PLAN_FIELDS = ("slot_expert", "quota", "host_ptr", "host_rank", "host_pslot",
               "reroute", "stats")

_lib = None
_P = ctypes.c_void_p


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                f"{LIB_PATH} is not built; run __graft_entry__.build() first")
        L = ctypes.CDLL(LIB_PATH)
        i32, i64, sz = ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
        gp, pp = ctypes.POINTER(Group), ctypes.POINTER(PlanBuf)
        L.ultraep_plan_sizes.argtypes = [gp, ctypes.POINTER(sz)]
        L.ultraep_count.argtypes = [_P, i64, i32, i32, i32, _P, _P, _P]
        L.ultraep_plan.argtypes = [_P, gp, pp, _P, sz, _P]
        L.ultraep_plan_noalloc.argtypes = [_P, gp, pp, _P]
        L.ultraep_plan_replicate.argtypes = [_P, gp, pp, _P, sz, _P]
        L.ultraep_plan_reroute.argtypes = [_P, gp, pp, _P]
        L.ultraep_plan_ws_bytes.argtypes = [gp]
        L.ultraep_plan_ws_bytes.restype = sz
        L.ultraep_dispatch_ws_bytes.argtypes = [i64, i32, gp]
        L.ultraep_dispatch_ws_bytes.restype = sz
        L.ultraep_dispatch.argtypes = [_P, _P, i64, i32, i32, i32, gp, pp, _P,
                                       _P, _P, _P, sz, _P, _P]
        L.ultraep_dispatch_layout.argtypes = [_P, i64, i32, i32, gp, pp, _P, _P,
                                              _P, sz, _P, _P]
        L.ultraep_dispatch_scatter.argtypes = [_P, i64, i32, i32, _P, _P, _P, _P]
        L.ultraep_pack_replicas.argtypes = [_P, i64, i32, gp, pp, _P, i64, _P,
                                            _P, _P]
        L.ultraep_reroute_and_pack.argtypes = [_P, gp, pp, _P, i64, i32, _P, i64, _P,
                                               _P, _P]
        L.ultraep_relay_plan.argtypes = [gp, pp, i32, _P, _P, _P, _P, _P]
        L.ultraep_pack_relay.argtypes = [_P, _P, i64, i32, gp, pp, _P, _P, i64, _P,
                                         _P, _P]
        L.ultraep_combine.argtypes = [_P, i64, _P, _P, i64, i32, i32, _P, _P, _P]
        L.ultraep_grad_reduce.argtypes = [_P, _P, i64, i32, gp, pp, i64, _P, _P]
        L.ultraep_strerror.argtypes = [ctypes.c_int]
        L.ultraep_strerror.restype = ctypes.c_char_p
        for f in ("ultraep_plan_sizes", "ultraep_count", "ultraep_plan",
                  "ultraep_plan_noalloc", "ultraep_plan_replicate", "ultraep_plan_reroute",
                  "ultraep_dispatch", "ultraep_dispatch_layout",
                  "ultraep_dispatch_scatter", "ultraep_pack_replicas",
                  "ultraep_reroute_and_pack", "ultraep_relay_plan",
                  "ultraep_pack_relay", "ultraep_combine", "ultraep_grad_reduce"):
            getattr(L, f).restype = ctypes.c_int
        _lib = L
    return _lib


def ultraep_strerror(code: int) -> str:
    return lib().ultraep_strerror(int(code)).decode()


def _check(rc, where):
    if rc != ULTRAEP_OK:
        raise UltraEPError(rc, where)
    return rc


def _ptr(t):
    """Device address of a torch tensor (None for None / empty tensors)."""
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("expected a device tensor")
    if not t.is_contiguous():
        raise ValueError("expected a contiguous tensor")
    return t.data_ptr() if t.numel() else None


def _need(t, n, esize, name):
    """Raises unless t holds at least n elements of esize bytes, so that no
    kernel reads or writes past a caller's tensor (n <= 0 needs nothing)."""
    if n <= 0:
        return
    if t is None:
        raise ValueError(f"{name}: a device tensor of {n} elements is needed")
    if t.element_size() != esize:
        raise ValueError(f"{name}: expected {esize}-byte elements, got {t.dtype}")
    if t.numel() < n:
        raise ValueError(f"{name}: needs {n} elements, has {t.numel()}")


def _stream(stream):
    if stream is not None:
        return stream.cuda_stream if hasattr(stream, "cuda_stream") else stream
    import torch
    return torch.cuda.current_stream().cuda_stream


def ultraep_plan_sizes(g: Group):
    out = (ctypes.c_size_t * 7)()
    _check(lib().ultraep_plan_sizes(ctypes.byref(g), out), "ultraep_plan_sizes")
    return tuple(int(v) for v in out)


class Plan:
    """Device buffers of one plan (torch tensors), their C descriptor, and the
    planner's device workspace."""

    def __init__(self, g: Group, device="cuda"):
        import torch
        n = ultraep_plan_sizes(g)
        dt = [torch.int32] * 6 + [torch.int64]
        for name, cnt, d in zip(PLAN_FIELDS, n, dt):
            setattr(self, name, torch.empty(cnt, dtype=d, device=device))
        self.g = g
        self.c = PlanBuf(*[_ptr(getattr(self, f)) for f in PLAN_FIELDS])
        self.ws = torch.empty(ultraep_plan_ws_bytes(g), dtype=torch.uint8,
                              device=device)


def ultraep_count(topk, T, k, E, n_groups, counts, status, stream=None):
    _need(topk, n_groups * T * k, 4, "topk")
    _need(counts, n_groups * E, 4, "counts")
    _need(status, 1, 4, "status")
    return _check(lib().ultraep_count(_ptr(topk), T, k, E, n_groups,
                                      _ptr(counts), _ptr(status),
                                      _stream(stream)), "ultraep_count")


def ultraep_plan_ws_bytes(g: Group) -> int:
    return int(lib().ultraep_plan_ws_bytes(ctypes.byref(g)))


def ultraep_plan(load, g: Group, plan: Plan, ws=None, stream=None):
    """ws: device workspace (defaults to the one the Plan object holds)."""
    ws = plan.ws if ws is None else ws
    _need(load, g.R * g.E, 4, "load")
    return _check(lib().ultraep_plan(_ptr(load), ctypes.byref(g),
                                     ctypes.byref(plan.c), _ptr(ws),
                                     ws.numel() * ws.element_size(),
                                     _stream(stream)), "ultraep_plan")


def ultraep_plan_noalloc(load, g: Group, plan: Plan, stream=None):
    """ultraep_plan with the library's fixed per-device workspace (plan.ws is
    not used); calls on one device must not overlap in time."""
    _need(load, g.R * g.E, 4, "load")
    return _check(lib().ultraep_plan_noalloc(_ptr(load), ctypes.byref(g),
                                             ctypes.byref(plan.c), _stream(stream)),
                  "ultraep_plan_noalloc")


def ultraep_plan_replicate(load, g: Group, plan: Plan, ws=None, stream=None):
    ws = plan.ws if ws is None else ws
    _need(load, g.R * g.E, 4, "load")
    return _check(lib().ultraep_plan_replicate(
        _ptr(load), ctypes.byref(g), ctypes.byref(plan.c), _ptr(ws),
        ws.numel() * ws.element_size(), _stream(stream)), "ultraep_plan_replicate")


def ultraep_plan_reroute(load, g: Group, plan: Plan, stream=None):
    _need(load, g.R * g.E, 4, "load")
    return _check(lib().ultraep_plan_reroute(
        _ptr(load), ctypes.byref(g), ctypes.byref(plan.c), _stream(stream)),
        "ultraep_plan_reroute")


def ultraep_dispatch_ws_bytes(T, k, g: Group) -> int:
    return int(lib().ultraep_dispatch_ws_bytes(T, k, ctypes.byref(g)))


def _layout_need(topk, T, k, g, row_of_slot, block_off, status):
    _need(topk, T * k, 4, "topk")
    _need(row_of_slot, T * k, 4, "row_of_slot")
    _need(block_off, g.R * g.S + 1, 8, "block_off")
    _need(status, 1, 4, "status")


def ultraep_dispatch(x, topk, T, k, H, rank, g: Group, plan: Plan, send,
                     row_of_slot, block_off, ws, status, stream=None):
    _need(x, T * H, 2, "x")
    _need(send, T * k * H, 2, "send")
    _layout_need(topk, T, k, g, row_of_slot, block_off, status)
    return _check(lib().ultraep_dispatch(
        _ptr(x), _ptr(topk), T, k, H, rank, ctypes.byref(g),
        ctypes.byref(plan.c), _ptr(send), _ptr(row_of_slot), _ptr(block_off),
        _ptr(ws), ws.numel() * ws.element_size(), _ptr(status),
        _stream(stream)), "ultraep_dispatch")


def ultraep_dispatch_layout(topk, T, k, rank, g: Group, plan: Plan,
                            row_of_slot, block_off, ws, status, stream=None):
    _layout_need(topk, T, k, g, row_of_slot, block_off, status)
    return _check(lib().ultraep_dispatch_layout(
        _ptr(topk), T, k, rank, ctypes.byref(g), ctypes.byref(plan.c),
        _ptr(row_of_slot), _ptr(block_off), _ptr(ws),
        ws.numel() * ws.element_size(), _ptr(status), _stream(stream)),
        "ultraep_dispatch_layout")


def ultraep_dispatch_scatter(x, T, k, H, row_of_slot, n_routed, send,
                             stream=None):
    """n_routed: a one-element int64 device tensor (e.g. block_off[-1:])."""
    _need(x, T * H, 2, "x")
    _need(row_of_slot, T * k, 4, "row_of_slot")
    _need(n_routed, 1 if T > 0 else 0, 8, "n_routed")
    _need(send, T * k * H, 2, "send")
    return _check(lib().ultraep_dispatch_scatter(
        _ptr(x), T, k, H, _ptr(row_of_slot), _ptr(n_routed), _ptr(send),
        _stream(stream)), "ultraep_dispatch_scatter")


def _pack_need(w_main, W, g, staging, cap, dest_off, status):
    _need(w_main, g.n_main * W, 2, "w_main")
    _need(staging, cap * W, 2, "staging")
    _need(dest_off, g.R + 1, 8, "dest_off")
    _need(status, 1, 4, "status")


def ultraep_pack_replicas(w_main, W, rank, g: Group, plan: Plan, staging, cap,
                          dest_off, status, stream=None):
    _pack_need(w_main, W, g, staging, cap, dest_off, status)
    return _check(lib().ultraep_pack_replicas(
        _ptr(w_main), W, rank, ctypes.byref(g), ctypes.byref(plan.c),
        _ptr(staging), cap, _ptr(dest_off), _ptr(status), _stream(stream)),
        "ultraep_pack_replicas")


def ultraep_reroute_and_pack(load, g: Group, plan: Plan, w_main, W, rank, staging,
                             cap, dest_off, status, stream=None):
    _need(load, g.R * g.E, 4, "load")
    _pack_need(w_main, W, g, staging, cap, dest_off, status)
    return _check(lib().ultraep_reroute_and_pack(
        _ptr(load), ctypes.byref(g), ctypes.byref(plan.c), _ptr(w_main), W, rank,
        _ptr(staging), cap, _ptr(dest_off), _ptr(status), _stream(stream)),
        "ultraep_reroute_and_pack")


def ultraep_relay_plan(g: Group, plan: Plan, threshold, slot_src, send_vol,
                       relay_stats, status, stream=None):
    _need(slot_src, g.R * g.n_slot, 4, "slot_src")
    _need(send_vol, g.R, 4, "send_vol")
    _need(relay_stats, 4, 8, "relay_stats")
    _need(status, 1, 4, "status")
    return _check(lib().ultraep_relay_plan(
        ctypes.byref(g), ctypes.byref(plan.c), threshold, _ptr(slot_src),
        _ptr(send_vol), _ptr(relay_stats), _ptr(status), _stream(stream)),
        "ultraep_relay_plan")


def ultraep_pack_relay(w_main, relay_src, W, rank, g: Group, plan: Plan, slot_src,
                       staging, cap, dest_off, status, stream=None):
    _pack_need(w_main, W, g, staging, cap, dest_off, status)
    _need(relay_src, g.n_slot * W, 2, "relay_src")
    _need(slot_src, g.R * g.n_slot, 4, "slot_src")
    return _check(lib().ultraep_pack_relay(
        _ptr(w_main), _ptr(relay_src), W, rank, ctypes.byref(g), ctypes.byref(plan.c),
        _ptr(slot_src), _ptr(staging), cap, _ptr(dest_off), _ptr(status),
        _stream(stream)), "ultraep_pack_relay")


def ultraep_combine(y, n_rows, gate, row_of_slot, T, k, H, out, status, stream=None):
    _need(y, n_rows * H, 2, "y")
    _need(gate, T * k, 4, "gate")
    _need(row_of_slot, T * k, 4, "row_of_slot")
    _need(out, T * H, 2, "out")
    _need(status, 1, 4, "status")
    return _check(lib().ultraep_combine(
        _ptr(y), n_rows, _ptr(gate), _ptr(row_of_slot), T, k, H, _ptr(out), _ptr(status),
        _stream(stream)), "ultraep_combine")


def ultraep_grad_reduce(main_grad, rgrad, W, rank, g: Group, plan: Plan, cap, status,
                        stream=None):
    _need(main_grad, g.n_main * W, 4, "main_grad")
    _need(rgrad, cap * W, 4, "rgrad")
    _need(status, 1, 4, "status")
    return _check(lib().ultraep_grad_reduce(
        _ptr(main_grad), _ptr(rgrad), W, rank, ctypes.byref(g), ctypes.byref(plan.c), cap,
        _ptr(status), _stream(stream)), "ultraep_grad_reduce")


def build():
    """Compile libultraep.so for gfx950 in-tree."""
    from . import _build
    global _lib
    _lib = None
    return _build.build()
