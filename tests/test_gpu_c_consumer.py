"""The library called from plain C (tests/native/abi_consumer.c, built by
__graft_entry__.build() against include/ultraep.h): count, plan, dispatch and
packing of one rank through raw hipMalloc pointers on the null stream, with
no torch in the process, equal the oracle byte for byte.  Needs an MI355X."""
import os
import subprocess
import tempfile

import numpy as np
import pytest

import gen
import oracle

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
EXE = os.path.join(ROOT, "tests", "native", "_build", "abi_consumer")


def _cases():
    c = gen.config(1)  # the tiny workload: 4 ranks, 16 experts, 2 slots, 512 tokens, top-2
    yield c.R, c.E, c.n_slot, c.T, c.k, c.u_min, c.beta_num, c.beta_den, gen.topk_all(c, 0)
    rng = np.random.default_rng(5)
    R, E, NS, T, k = 16, 64, 2, 700, 4
    p = rng.dirichlet(np.full(E, 0.3))
    yield R, E, NS, T, k, 8, 101, 100, rng.choice(E, (R, T, k), p=p).astype(np.int32)


@pytest.mark.parametrize("case", range(2))
def test_c_caller_matches_oracle(case):
    assert os.path.exists(EXE), "run __graft_entry__.build() first"
    R, E, NS, T, k, u_min, bn, bd, tk = list(_cases())[case]
    rng = np.random.default_rng(100 + case)
    H, W = 40, 264
    nm, V, S, cap = E // R, T * k, E // R + NS, R * NS
    og = oracle.Group(R, E, NS, u_min, bn, bd)
    load, st = oracle.count(tk, E, R)
    assert st == 0
    op = oracle.plan(load, og)
    X = op.slot_expert.reshape(R, NS)
    rank = int(np.argmax([((X >= 0) & (X // nm == r)).sum() for r in range(R)]))
    x = rng.integers(0, 1 << 16, (T, H)).astype(np.uint16)
    w = rng.integers(0, 1 << 16, (nm, W)).astype(np.uint16)
    with tempfile.TemporaryDirectory() as d:
        fin, fout = os.path.join(d, "in.bin"), os.path.join(d, "out.bin")
        with open(fin, "wb") as f:
            np.array([R, E, NS, T, k, H, W, rank, u_min, bn, bd], np.int64).tofile(f)
            np.ascontiguousarray(tk, np.int32).tofile(f)
            x.tofile(f)
            w.tofile(f)
        print(f"C caller: case {case} R={R} E={E} T={T} k={k} rank={rank}", flush=True)
        r = subprocess.run([EXE, fin, fout], capture_output=True, text=True, timeout=120)
        assert r.returncode == 0, r.stderr
        buf = open(fout, "rb").read()
    off = 0

    def take(dtype, n):
        nonlocal off
        a = np.frombuffer(buf, dtype, n, off)
        off += a.nbytes
        return a

    ncol = E + R * NS
    assert take(np.int32, 1)[0] == 0
    assert np.array_equal(take(np.int32, R * E), load.reshape(-1))
    for name, dt, n in [("slot_expert", np.int32, R * NS), ("quota", np.int32, E * R),
                        ("host_ptr", np.int32, E + 1), ("host_rank", np.int32, ncol),
                        ("host_pslot", np.int32, ncol), ("reroute", np.int32, R * ncol),
                        ("stats", np.int64, 8)]:
        assert np.array_equal(take(dt, n), getattr(op, name).reshape(-1)), name
    osend, oros, oboff, ost = oracle.dispatch(x, tk[rank], rank, og, op)
    assert ost == 0
    assert np.array_equal(take(np.uint16, V * H), osend.reshape(-1)), "send"
    assert np.array_equal(take(np.int32, V), oros), "row_of_slot"
    assert np.array_equal(take(np.int64, R * S + 1), oboff), "block_off"
    ostg, odoff, n_out, ost = oracle.pack(w, rank, og, op, cap)
    assert ost == 0
    assert np.array_equal(take(np.int64, R + 1), odoff), "dest_off"
    assert take(np.int64, 1)[0] == n_out > 0
    assert np.array_equal(take(np.uint16, n_out * W), ostg[:n_out].reshape(-1)), "staging"
    assert off == len(buf)
