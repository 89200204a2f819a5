"""Independent checks of what the paper fixes about a plan, a dispatch layout
and a pack, written from the definitions (Table 1, Sec. 4.3 constraints,
Sec. 5.2) rather than from the oracle's code.  Used on the oracle's outputs
(to pin it) and on the HIP library's outputs (on top of byte parity).
"""
from __future__ import annotations

import numpy as np


def hosts_of(g, p, e):
    a, b = int(p.host_ptr[e]), int(p.host_ptr[e + 1])
    return [int(t) for t in p.host_rank[a:b]], [int(s) for s in p.host_pslot[a:b]], a


def check_plan(load, g, p, *, check_locality=True):
    """I2-I6, I8, I9 plus CSR consistency.  Returns the per-rank loads after."""
    load = np.asarray(load, np.int64)
    R, E, NS, nm = g.R, g.E, g.n_slot, g.E // g.R
    X = np.asarray(p.slot_expert).reshape(R, NS)
    U = np.asarray(p.quota, np.int64).reshape(E, R)
    Q = np.asarray(p.reroute, np.int64).reshape(R, g.ncol)
    lam_e = load.sum(0)
    assert p.status == 0 and int(p.stats[6]) == 0

    # I2: quotas of every expert sum to its load
    assert np.array_equal(U.sum(1), lam_e), "I2"
    assert (U >= 0).all()

    # I4: slot capacity, no duplicates, no replica on the home rank,
    #     slots filled from index 0 upwards
    for t in range(R):
        row = [int(e) for e in X[t] if e >= 0]
        assert all(X[t, s] >= 0 for s in range(len(row))), "slots not packed"
        assert len(set(row)) == len(row), "I4 duplicate"
        assert all(e // nm != t for e in row), "I4 replica on home"
        assert all(0 <= e < E for e in row)

    # CSR: H(e) = home first, then the replica ranks ascending; pslots match X
    assert p.host_ptr[0] == 0
    total = int(p.host_ptr[E])
    assert (p.host_rank[total:] == -1).all() and (p.host_pslot[total:] == -1).all()
    n_rep = 0
    for e in range(E):
        H, P, j0 = hosts_of(g, p, e)
        assert H[0] == e // nm and P[0] == e - (e // nm) * nm
        assert H[1:] == sorted(H[1:]) and len(set(H)) == len(H)
        for t, ps in zip(H[1:], P[1:]):
            assert X[t, ps - nm] == e
        n_rep += len(H) - 1
        # I3: positive quota only on hosts
        others = [t for t in range(R) if t not in H]
        assert (U[e, others] == 0).all(), "I3"
        # I5: every replica carries at least u_min
        for t in H[1:]:
            assert U[e, t] >= g.u_min, "I5"
    assert n_rep == int((X >= 0).sum()) == int(p.stats[4])

    # I6: every rank ends within tau*, and tau* within the initial bracket
    after = U.sum(0)
    tau = int(p.stats[0])
    assert after.max(initial=0) <= tau <= int(p.stats[2]), "I6"

    # I8: margins of the reroute split (exact)
    assert (Q >= 0).all()
    assert (Q[:, total:] == 0).all()
    for e in range(E):
        H, P, j0 = hosts_of(g, p, e)
        blk = Q[:, j0:j0 + len(H)]
        assert np.array_equal(blk.sum(1), load[:, e]), "I8 rows"
        assert np.array_equal(blk.sum(0), U[e, H]), "I8 cols"
        # I9: locality first
        if check_locality:
            for i, t in enumerate(H):
                assert blk[t, i] == min(load[t, e], U[e, t]), "I9"
    return after


def check_dispatch(x, topk, rank, g, p, send, ros, boff):
    """I10/I11: block sizes are the plan's q, rows form a bijection onto the
    routed slots, blocks keep token order, every row is a bit copy, and the
    k-th local token of (rank, e) goes to the instance whose cumulative quota
    first exceeds its ordinal."""
    R, E, nm, S = g.R, g.E, g.E // g.R, g.E // g.R + g.n_slot
    Q = np.asarray(p.reroute, np.int64).reshape(R, g.ncol)[rank]
    X = np.asarray(p.slot_expert).reshape(R, g.n_slot)
    flat = np.asarray(topk).reshape(-1)
    k = np.asarray(topk).shape[-1]
    V = flat.size
    valid = flat >= 0
    nv = int(valid.sum())
    # block sizes
    cnt = np.zeros(R * S, np.int64)
    for t in range(R):
        for ps in range(S):
            e = t * nm + ps if ps < nm else int(X[t, ps - nm])
            if e < 0:
                continue
            H, P, j0 = hosts_of(g, p, e)
            i = [ii for ii, (tt, pp) in enumerate(zip(H, P)) if tt == t and pp == ps]
            assert len(i) == 1
            cnt[t * S + ps] = Q[j0 + i[0]]
    assert boff[0] == 0 and np.array_equal(np.diff(boff), cnt)
    assert boff[-1] == nv
    # bijection
    rows = ros[valid]
    assert (ros[~valid] == -1).all()
    assert np.array_equal(np.sort(rows), np.arange(nv))
    # per expert: slots in flat order split into consecutive runs by q
    for e in range(E):
        idx = np.nonzero(flat == e)[0]
        H, P, j0 = hosts_of(g, p, e)
        c0 = 0
        for i, (t, ps) in enumerate(zip(H, P)):
            q = int(Q[j0 + i])
            run = idx[c0:c0 + q]
            start = int(boff[t * S + ps])
            assert np.array_equal(ros[run], start + np.arange(q))
            c0 += q
        assert c0 == idx.size
    # bit copies and zero tail
    xs = np.asarray(x)
    send = np.asarray(send).reshape(V, xs.shape[1])
    vi = np.nonzero(valid)[0]
    assert np.array_equal(send[ros[vi]], xs[vi // k])
    assert (send[nv:] == 0).all()


def check_pack(w_main, rank, g, p, staging, doff, n_out):
    """I12: staging holds bit copies of the right main experts, in
    (destination rank, destination slot) order."""
    R, NS, nm = g.R, g.n_slot, g.E // g.R
    X = np.asarray(p.slot_expert).reshape(R, NS)
    ents = [(t, s, int(X[t, s])) for t in range(R) for s in range(NS)
            if X[t, s] >= 0 and X[t, s] // nm == rank]
    assert n_out == len(ents)
    for t in range(R + 1):
        assert doff[t] == sum(1 for (tt, _, _) in ents if tt < t)
    for n, (_, _, e) in enumerate(ents):
        assert np.array_equal(staging[n], w_main[e - rank * nm])
