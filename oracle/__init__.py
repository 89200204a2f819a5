"""UltraEP reference oracle (ctypes wrapper) — TEST INFRASTRUCTURE ONLY.

The oracle is a plain, slow, single-threaded C implementation of the paper's
definitions (Algorithm 1, Sec. 5.1-5.2, Sec. 6.1 of arXiv 2606.04101).  Only
the test-suite, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this module; the product library never does.

Every function takes and returns numpy arrays (host memory).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_BUILT = os.path.join(_HERE, "liboracle.so")
# ULTRAEP_ORACLE_LIB names another build of oracle.c (the sanitizer test's)
_LIB = os.environ.get("ULTRAEP_ORACLE_LIB") or _BUILT

OK, EINVAL, ENOSPC, EDATA, ELEMMA = 0, -1, -2, -4, -6


def build() -> str:
    """Compile ``liboracle.so`` with gcc (-O2, C11, no GPU headers)."""
    # -ffp-contract=off: no fused multiply-add in the fp32 combine and
    # reduction (each product and sum rounds on its own)
    cmd = ["gcc", "-O2", "-std=c11", "-Wall", "-Wextra", "-ffp-contract=off",
           "-fPIC", "-shared", "-o", _BUILT + ".tmp", _SRC]
    subprocess.run(cmd, check=True, cwd=_HERE)
    os.replace(_BUILT + ".tmp", _BUILT)
    return _BUILT


class _Group(ctypes.Structure):
    _fields_ = [("R", ctypes.c_int32), ("E", ctypes.c_int32),
                ("n_slot", ctypes.c_int32), ("u_min", ctypes.c_int64),
                ("beta_num", ctypes.c_int32), ("beta_den", ctypes.c_int32)]


@dataclass(frozen=True)
class Group:
    """EP group metadata: R ranks, E experts, n_slot redundant slots per rank,
    quota floor u_min and balancing target beta = beta_num / beta_den."""
    R: int
    E: int
    n_slot: int
    u_min: int
    beta_num: int = 101
    beta_den: int = 100

    @property
    def n_main(self) -> int:
        return self.E // self.R

    @property
    def S(self) -> int:
        return self.n_main + self.n_slot

    @property
    def ncol(self) -> int:
        return self.E + self.R * self.n_slot

    def c(self) -> _Group:
        return _Group(self.R, self.E, self.n_slot, self.u_min, self.beta_num,
                      self.beta_den)


_lib = None
_P = ctypes.c_void_p


def _load(path):
    L = ctypes.CDLL(path)
    i32, i64 = ctypes.c_int32, ctypes.c_int64
    gp = ctypes.POINTER(_Group)
    L.orc_count.argtypes = [_P, i64, i32, i32, i32, _P]
    L.orc_probe.argtypes = [_P, gp, i64, _P, _P, _P]
    L.orc_plan.argtypes = [_P, gp, i32, _P, _P, _P, _P, _P, _P, _P]
    L.orc_bisect_trace.argtypes = [_P, gp, _P, _P, i32]
    L.orc_apportion.argtypes = [i64, _P, i32, _P]
    L.orc_dispatch.argtypes = [_P, _P, i64, i32, i32, i32, gp, _P, _P, _P,
                               _P, _P, _P, _P, _P]
    L.orc_pack.argtypes = [_P, i64, i32, gp, _P, _P, i64, _P, _P]
    L.orc_metrics.argtypes = [_P, gp, _P, _P, _P, _P, _P]
    L.orc_relay.argtypes = [gp, _P, _P, _P, _P, i32, _P, _P, _P]
    L.orc_pack_relay.argtypes = [_P, _P, i64, i32, gp, _P, _P, _P, i64, _P, _P]
    L.orc_combine.argtypes = [_P, _P, _P, i64, i32, i32, i64, _P]
    L.orc_grad_reduce.argtypes = [_P, _P, i64, i32, gp, _P, i64, _P]
    for f in ("orc_count", "orc_probe", "orc_plan", "orc_bisect_trace",
              "orc_apportion", "orc_dispatch", "orc_pack", "orc_metrics",
              "orc_relay", "orc_pack_relay", "orc_combine", "orc_grad_reduce"):
        getattr(L, f).restype = ctypes.c_int
    return L


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        _lib = _load(_LIB)
    return _lib


def use_library(path):
    """Point this wrapper at another build of oracle.c (mutation tests);
    ``None`` restores the default build.  Returns the previous handle."""
    global _lib
    prev = _lib
    _lib = None if path is None else _load(path)
    return prev


def _p(a):
    return None if a is None else a.ctypes.data_as(_P)


def _c(a, dt):
    return np.ascontiguousarray(a, dtype=dt)


def count(topk, E, n_groups=1):
    """counts[g, e] = number of (token, k) slots of group g routed to e."""
    topk = _c(topk, np.int32)
    per = topk.size // n_groups
    k = topk.shape[-1] if topk.ndim > 1 else 1
    T = per // k
    counts = np.zeros((n_groups, E), np.int32)
    st = lib().orc_count(_p(topk), T, k, E, n_groups, _p(counts))
    return counts, st


def probe(load, g: Group, tau):
    """One greedy feasibility probe at threshold tau -> (feasible, Ut, X, st)."""
    load = _c(load, np.int32)
    feas = np.zeros(1, np.int32)
    Ut = np.zeros((g.E, g.R), np.int64)
    X = np.full((g.R, max(g.n_slot, 0)), -1, np.int32)
    gc = g.c()
    st = lib().orc_probe(_p(load), ctypes.byref(gc), int(tau), _p(feas),
                         _p(Ut), _p(X) if g.n_slot > 0 else None)
    return bool(feas[0]), Ut, X, st


@dataclass
class Plan:
    slot_expert: np.ndarray  # [R, n_slot]
    quota: np.ndarray        # [E, R]
    host_ptr: np.ndarray     # [E+1]
    host_rank: np.ndarray    # [ncol]
    host_pslot: np.ndarray   # [ncol]
    reroute: np.ndarray      # [R, ncol]
    stats: np.ndarray        # [8]
    status: int

    @property
    def tau_star(self):
        return int(self.stats[0])


def plan(load, g: Group, locality=True) -> Plan:
    load = _c(load, np.int32)
    assert load.shape == (g.R, g.E)
    ns = max(g.n_slot, 0)
    ncol = g.E + g.R * ns
    # poisoned outputs: orc_plan must write every element, padding included
    X = np.full((g.R, ns), -7, np.int32)
    U = np.full((g.E, g.R), -7, np.int32)
    hp = np.full(g.E + 1, -7, np.int32)
    hr = np.full(ncol, -7, np.int32)
    hs = np.full(ncol, -7, np.int32)
    q = np.full((g.R, ncol), -7, np.int32)
    stats = np.full(8, -7, np.int64)
    gc = g.c()
    st = lib().orc_plan(_p(load), ctypes.byref(gc), int(bool(locality)),
                        _p(X) if X.size else _p(np.zeros(1, np.int32)),
                        _p(U), _p(hp), _p(hr), _p(hs), _p(q), _p(stats))
    return Plan(X, U, hp, hr, hs, q, stats, st)


def bisect_trace(load, g: Group, cap=128):
    load = _c(load, np.int32)
    taus = np.zeros(cap, np.int64)
    feas = np.zeros(cap, np.int32)
    gc = g.c()
    n = lib().orc_bisect_trace(_p(load), ctypes.byref(gc), _p(taus), _p(feas),
                               cap)
    assert n >= 0, n
    n = min(n, cap)
    return [(int(taus[i]), bool(feas[i])) for i in range(n)]


def apportion(demand, ures):
    ures = _c(ures, np.int64)
    out = np.zeros(ures.size, np.int64)
    st = lib().orc_apportion(int(demand), _p(ures), ures.size, _p(out))
    assert st == OK, st
    return out


def dispatch(x, topk, rank, g: Group, p: Plan, poison=True):
    """-> send [T*k, H] uint16, row_of_slot [T*k], block_off [R*S+1], status.
    poison: hand orc_dispatch outputs filled with a pattern it must overwrite
    (every row_of_slot entry, every block offset, every send row: the routed
    rows and the zero tail), so a missed write shows; False hands it zeroed
    buffers (the timed baseline, where filling 2 bytes per send element would
    add host work the oracle itself does not do)."""
    x = _c(x, np.uint16)
    topk = _c(topk, np.int32)
    T, H = x.shape
    k = topk.shape[1] if topk.ndim == 2 else 1
    if poison:
        send = np.full((T * k, H), 0xDEAD, np.uint16)
        ros = np.full(T * k, -7, np.int32)
        boff = np.full(g.R * g.S + 1, -7, np.int64)
    else:
        send = np.zeros((T * k, H), np.uint16)
        ros = np.full(T * k, -1, np.int32)
        boff = np.zeros(g.R * g.S + 1, np.int64)
    gc = g.c()
    X = p.slot_expert if p.slot_expert.size else np.zeros(1, np.int32)
    st = lib().orc_dispatch(_p(x), _p(topk), T, k, H, rank, ctypes.byref(gc),
                            _p(X), _p(p.host_ptr), _p(p.host_rank),
                            _p(p.host_pslot), _p(p.reroute), _p(send), _p(ros),
                            _p(boff))
    return send, ros, boff, st


def pack(w_main, rank, g: Group, p: Plan, cap):
    """-> staging [cap, W] uint16 (first n_out entries), dest_off [R+1], n_out, st"""
    w_main = _c(w_main, np.uint16)
    W = w_main.shape[1]
    staging = np.zeros((max(cap, 0), W), np.uint16)
    doff = np.zeros(g.R + 1, np.int64)
    n_out = np.zeros(1, np.int64)
    gc = g.c()
    X = p.slot_expert if p.slot_expert.size else np.zeros(1, np.int32)
    st = lib().orc_pack(_p(w_main), W, rank, ctypes.byref(gc), _p(X),
                        _p(staging) if staging.size else None, cap, _p(doff),
                        _p(n_out))
    return staging, doff, int(n_out[0]), st


@dataclass
class Relay:
    slot_src: np.ndarray   # [R, n_slot] sender rank of each redundant slot, -1 empty
    send_vol: np.ndarray   # [R] blobs sent per rank
    stats: np.ndarray      # [4] relay experts, relays, max volume before / after
    status: int


def relay(g: Group, p, threshold=4) -> Relay:
    """Relay trees (Sec. 6.2) of a plan; p needs slot_expert, host_ptr,
    host_rank and host_pslot."""
    ns = max(g.n_slot, 0)
    X = _c(p.slot_expert, np.int32).reshape(-1)
    src = np.full(max(g.R * ns, 1), -7, np.int32)
    vol = np.full(g.R, -7, np.int32)
    stats = np.zeros(4, np.int64)
    gc = g.c()
    st = lib().orc_relay(ctypes.byref(gc), _p(X) if X.size else _p(np.zeros(1, np.int32)),
                         _p(_c(p.host_ptr, np.int32)), _p(_c(p.host_rank, np.int32)),
                         _p(_c(p.host_pslot, np.int32)), int(threshold), _p(src),
                         _p(vol), _p(stats))
    return Relay(src[: g.R * ns].reshape(g.R, ns), vol, stats, st)


def pack_relay(w_main, relay_src, rank, g: Group, slot_expert, slot_src, cap):
    """-> staging [cap, W] uint16 (first n_out entries), dest_off [R+1], n_out, st"""
    w_main = _c(w_main, np.uint16)
    W = w_main.shape[1]
    rs = None if relay_src is None else _c(relay_src, np.uint16)
    staging = np.zeros((max(cap, 0), W), np.uint16)
    doff = np.zeros(g.R + 1, np.int64)
    n_out = np.zeros(1, np.int64)
    gc = g.c()
    X = _c(slot_expert, np.int32).reshape(-1)
    S = _c(slot_src, np.int32).reshape(-1)
    z = np.zeros(1, np.int32)
    st = lib().orc_pack_relay(_p(w_main), _p(rs), W, rank, ctypes.byref(gc),
                              _p(X) if X.size else _p(z), _p(S) if S.size else _p(z),
                              _p(staging) if staging.size else None, cap, _p(doff),
                              _p(n_out))
    return staging, doff, int(n_out[0]), st


def combine(y, gate, row_of_slot):
    """-> out [T, H] uint16 (bf16 bits), status.  y [n_rows, H] uint16,
    gate [T, k] float32, row_of_slot [T*k] or [T, k] int32."""
    y = _c(y, np.uint16)
    gate = _c(gate, np.float32)
    T, k = gate.shape
    ros = _c(row_of_slot, np.int32).reshape(-1)
    n_rows, H = y.shape
    out = np.full((T, H), 0xDEAD, np.uint16)  # poisoned: every output row must be written
    st = lib().orc_combine(_p(y) if y.size else None, _p(gate), _p(ros), T, k, H, n_rows,
                           _p(out))
    return out, st


def grad_reduce(main_grad, rgrad, rank, g: Group, slot_expert, cap):
    """In place on copies: -> (main_grad', rgrad', n_out, status)."""
    mg = np.array(main_grad, dtype=np.float32, copy=True, order="C")
    rg = np.array(rgrad, dtype=np.float32, copy=True, order="C")
    W = mg.shape[1]
    n_out = np.zeros(1, np.int64)
    gc = g.c()
    X = _c(slot_expert, np.int32).reshape(-1)
    st = lib().orc_grad_reduce(_p(mg), _p(rg) if rg.size else None, W, rank,
                               ctypes.byref(gc), _p(X) if X.size else _p(np.zeros(1, np.int32)),
                               cap, _p(n_out))
    return mg, rg, int(n_out[0]), st


def metrics(load, g: Group, p: Plan):
    """-> dict of the Table 3 style diagnostics for a plan."""
    load = _c(load, np.int32)
    out = np.zeros(6, np.int64)
    gc = g.c()
    st = lib().orc_metrics(_p(load), ctypes.byref(gc), _p(p.quota),
                           _p(p.host_ptr), _p(p.host_rank), _p(p.reroute),
                           _p(out))
    assert st == OK, st
    before, L, after, n_rep, max_h, remote = (int(v) for v in out)
    mean = L / g.R if L else 0.0
    return {
        "imbalance_before": before / mean if mean else 1.0,
        "imbalance_after": after / mean if mean else 1.0,
        "n_replicas": n_rep,
        "max_hosts": max_h,
        "inflight_ratio": remote / L if L else 0.0,
        "max_load_before": before,
        "max_load_after": after,
        "total_load": L,
    }
