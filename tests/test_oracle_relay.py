"""Pins of the oracle's relay trees (Sec. 6.2, load-aware relay scheduling)
and of the packing that follows them.  The expected trees are derived by hand
from the paper's description and the readings stated in the oracle (relay
count = integer nearest sqrt(replicas), volumes in blobs, hot experts by
replica count descending, ties to the smaller rank); none is produced by the
oracle itself."""
import numpy as np
import pytest

import oracle


def csr_from_slots(R, E, NS, X):
    """host_ptr / host_rank / host_pslot of a slot map, written out here from
    the layout's definition (home first, then replica ranks ascending)."""
    nm = E // R
    X = np.asarray(X, np.int32).reshape(R, NS)
    hp = [0]
    hr, hs = [], []
    for e in range(E):
        hr.append(e // nm)
        hs.append(e - (e // nm) * nm)
        for t in range(R):
            for s in range(NS):
                if X[t, s] == e:
                    hr.append(t)
                    hs.append(nm + s)
        hp.append(len(hr))
    ncol = E + R * NS
    hr += [-1] * (ncol - len(hr))
    hs += [-1] * (ncol - len(hs))

    class P:
        pass
    p = P()
    p.slot_expert = X
    p.host_ptr = np.array(hp, np.int32)
    p.host_rank = np.array(hr, np.int32)
    p.host_pslot = np.array(hs, np.int32)
    return p


def one_hot_expert(f, R=None):
    """Expert 0 (home rank 0) replicated on ranks 1..f, one main expert and
    one redundant slot per rank."""
    R = R or f + 1
    X = np.full((R, 1), -1, np.int32)
    X[1:f + 1, 0] = 0
    g = oracle.Group(R, R, 1, 1)
    return g, csr_from_slots(R, R, 1, X)


def test_figure_nine_replicas_three_relays():
    """The relay figure of Sec. 6.2: one expert on rank 0 multicast to ranks
    1..9 uses three relays, so the source's fan-out drops from 9 to 3.  With
    every other rank idle the relays take two leaves each."""
    g, p = one_hot_expert(9)
    r = oracle.relay(g, p, threshold=4)
    assert r.status == oracle.OK
    src = r.slot_src[:, 0]
    relays = sorted(t for t in range(1, 10) if src[t] == 0)
    assert len(relays) == 3
    # reading: equal volumes tie to the smaller rank (the figure's choice of
    # ranks 2, 5, 8 is an illustration; the text fixes no tie-break)
    assert relays == [1, 2, 3]
    assert src.tolist() == [-1, 0, 0, 0, 1, 2, 3, 1, 2, 3]
    assert r.send_vol.tolist() == [3, 2, 2, 2, 0, 0, 0, 0, 0, 0]
    assert r.stats.tolist() == [1, 3, 9, 3]


# replica count f -> relays: the integer nearest sqrt(f), by hand
FRONTIER = {5: 2, 6: 2, 7: 3, 8: 3, 9: 3, 10: 3, 11: 3, 12: 3, 13: 4, 16: 4,
            20: 4, 21: 5, 30: 5, 31: 6, 42: 6, 43: 7, 56: 7, 57: 8, 63: 8}


@pytest.mark.parametrize("f,n", sorted(FRONTIER.items()))
def test_single_hot_expert_closed_form(f, n):
    """One hot expert, every other rank idle: n relays (the smallest ranks),
    the f - n leaves dealt round-robin over the relays in rank order, the
    source sends n blobs and relay i sends ceil((f - n - i) / n)."""
    g, p = one_hot_expert(f)
    r = oracle.relay(g, p, threshold=4)
    assert r.status == oracle.OK
    src = r.slot_src[:, 0]
    assert all(src[t] == 0 for t in range(1, n + 1))
    leaves = list(range(n + 1, f + 1))
    for i, t in enumerate(leaves):
        assert src[t] == 1 + i % n
    want = [n] + [-(-(f - n - i) // n) for i in range(n)] + [0] * (f - n)
    assert r.send_vol.tolist() == want
    assert r.stats.tolist() == [1, n, f, max(want)]


@pytest.mark.parametrize("f", [1, 2, 3, 4])
def test_at_most_four_replicas_no_relay(f):
    """The threshold is 4 and relays are built when the replica count
    exceeds it: up to 4 replicas every slot is served by the home rank."""
    g, p = one_hot_expert(f, R=8)
    r = oracle.relay(g, p, threshold=4)
    assert r.status == oracle.OK
    assert r.slot_src[:, 0].tolist() == [-1] + [0] * f + [-1] * (7 - f)
    assert r.send_vol.tolist() == [f] + [0] * 7
    assert r.stats.tolist() == [0, 0, f, f]


def test_relays_avoid_busy_senders():
    """Load awareness: rank 1 already sends expert 1 to three ranks and rank 2
    sends expert 2 once, so the relays of expert 0 (7 replicas, 3 relays) are
    the idle ranks 3, 4, 5; the leaves 1, 2, 6, 7 go to the least loaded
    relay at each step.  Derived by hand."""
    R, E, NS = 8, 8, 2
    X = np.full((R, NS), -1, np.int32)
    X[1:8, 0] = 0           # expert 0 on ranks 1..7
    X[2:5, 1] = 1           # expert 1 (home 1) on ranks 2, 3, 4
    X[5, 1] = 2             # expert 2 (home 2) on rank 5
    g = oracle.Group(R, E, NS, 1)
    r = oracle.relay(g, csr_from_slots(R, E, NS, X), threshold=4)
    assert r.status == oracle.OK
    assert r.slot_src[:, 0].tolist() == [-1, 3, 4, 0, 0, 0, 5, 3]
    assert r.slot_src[:, 1].tolist() == [-1, -1, 1, 1, 1, 2, -1, -1]
    assert r.send_vol.tolist() == [3, 3, 1, 2, 1, 1, 0, 0]
    assert r.stats.tolist() == [1, 3, 7, 3]


def test_second_hot_expert_sees_first_ones_volumes():
    """Two hot experts with 6 replicas each on ranks 1..6: expert 0 goes
    first (equal counts, smaller id), takes relays 1, 2 (two leaves each);
    expert 7 then avoids them and relays through 3, 4.  Derived by hand."""
    R, E, NS = 8, 8, 2
    X = np.full((R, NS), -1, np.int32)
    X[1:7, 0] = 0
    X[1:7, 1] = 7
    g = oracle.Group(R, E, NS, 1)
    r = oracle.relay(g, csr_from_slots(R, E, NS, X), threshold=4)
    assert r.status == oracle.OK
    assert r.slot_src[:, 0].tolist() == [-1, 0, 0, 1, 2, 1, 2, -1]
    assert r.slot_src[:, 1].tolist() == [-1, 3, 4, 7, 7, 3, 4, -1]
    assert r.send_vol.tolist() == [2, 2, 2, 2, 2, 0, 0, 2]
    assert r.stats.tolist() == [2, 4, 6, 2]


def test_larger_fanout_goes_first():
    """Expert 7 has 6 replicas and expert 0 has 5: expert 7 is processed
    first although its id is larger, so it takes the idle relays 1, 2 and
    expert 0 relays through 3, 4.  Derived by hand."""
    R, E, NS = 8, 8, 2
    X = np.full((R, NS), -1, np.int32)
    X[1:6, 0] = 0           # expert 0 on 1..5   (f = 5, 2 relays)
    X[1:7, 1] = 7           # expert 7 on 1..6   (f = 6, 2 relays)
    g = oracle.Group(R, E, NS, 1)
    r = oracle.relay(g, csr_from_slots(R, E, NS, X), threshold=4)
    assert r.status == oracle.OK
    # expert 7: relays 1, 2; leaves 3, 4, 5, 6 -> 1, 2, 1, 2
    assert r.slot_src[:, 1].tolist() == [-1, 7, 7, 1, 2, 1, 2, -1]
    # expert 0: volumes 1:2 2:2 3:0 4:0 5:0 -> relays 3, 4; leaves 1, 2, 5
    # -> 3, 4, 3
    assert r.slot_src[:, 0].tolist() == [-1, 3, 4, 0, 0, 3, -1, -1]
    assert r.send_vol.tolist() == [2, 2, 2, 2, 1, 0, 0, 2]


def _tree_invariants(g, p, rel, threshold):
    R, NS, nm = g.R, g.n_slot, g.n_main
    X = np.asarray(p.slot_expert).reshape(R, NS)
    src = rel.slot_src
    hp, hr = p.host_ptr, p.host_rank
    sends = np.zeros(R, np.int64)
    for t in range(R):
        for s in range(NS):
            e = X[t, s]
            if e < 0:
                assert src[t, s] == -1
                continue
            h = e // nm
            u = src[t, s]
            sends[u] += 1
            if u == h:
                continue
            # a relay hosts e and receives it from the home rank
            assert u in hr[hp[e] + 1:hp[e + 1]]
            su = [src[u, s2] for s2 in range(NS) if X[u, s2] == e]
            assert su == [h]
    assert np.array_equal(sends, rel.send_vol)
    assert rel.send_vol.sum() == (X >= 0).sum()
    n_hot, n_rel = 0, 0
    for e in range(g.E):
        f = hp[e + 1] - hp[e] - 1
        relays = {int(src[t, s]) for t in range(R) for s in range(NS)
                  if X[t, s] == e and src[t, s] != e // nm}
        if f > threshold:
            n_hot += 1
            n_rel += FRONTIER_OF(f)
            assert len(relays) <= FRONTIER_OF(f)
        else:
            assert not relays
    assert rel.stats[0] == n_hot and rel.stats[1] == n_rel


def FRONTIER_OF(f):
    n = int(np.floor(np.sqrt(f)))
    while (n + 1) ** 2 <= f:
        n += 1
    while n * n > f:
        n -= 1
    return n + 1 if f - n * n > n else n


@pytest.mark.parametrize("cid", [1, 2, 3, 4, 5])
@pytest.mark.parametrize("threshold", [0, 1, 2, 4])
def test_tree_invariants_on_workloads(cid, threshold):
    import gen
    c = gen.config(cid)
    g = oracle.Group(c.R, c.E, c.n_slot, c.u_min, c.beta_num, c.beta_den)
    load, _ = oracle.count(gen.topk_all(c, 0), c.E, c.R)
    p = oracle.plan(load, g)
    rel = oracle.relay(g, p, threshold)
    assert rel.status == oracle.OK
    _tree_invariants(g, p, rel, threshold)


def test_relay_rejects_inconsistent_plan():
    g, p = one_hot_expert(6)
    p.host_rank = p.host_rank.copy()
    p.host_rank[3], p.host_rank[4] = p.host_rank[4], p.host_rank[3]  # not ascending
    assert oracle.relay(g, p, 4).status == oracle.EDATA


def test_pack_relay_stages_for_the_slots_a_rank_sends():
    """Rank 1 relays expert 0 (figure case) to ranks 4 and 7: its staging
    holds two copies of its own slot's blob, ranks ascending; rank 0 sends
    its main expert to the three relays only."""
    g, p = one_hot_expert(9)
    rel = oracle.relay(g, p, 4)
    W = 40
    rng = np.random.default_rng(5)
    for rank, dests in [(0, [1, 2, 3]), (1, [4, 7]), (2, [5, 8]), (5, [])]:
        w = rng.integers(0, 1 << 16, (1, W), dtype=np.uint16)
        own = rng.integers(0, 1 << 16, (1, W), dtype=np.uint16)
        stg, doff, n, st = oracle.pack_relay(w, own, rank, g, p.slot_expert,
                                             rel.slot_src, 9)
        assert st == oracle.OK and n == len(dests)
        blob = w[0] if rank == 0 else own[0]
        for i in range(n):
            assert np.array_equal(stg[i], blob)
        want = [sum(1 for d in dests if d < t) for t in range(g.R)] + [n]
        assert doff.tolist() == want


def test_pack_relay_without_relays_is_the_plain_pack():
    """With no hot expert every slot is sent by its home rank, and the
    packing equals the one without relay trees on every rank."""
    import gen
    c = gen.config(1)
    g = oracle.Group(c.R, c.E, c.n_slot, c.u_min, c.beta_num, c.beta_den)
    load, _ = oracle.count(gen.topk_all(c, 0), c.E, c.R)
    p = oracle.plan(load, g)
    rel = oracle.relay(g, p, 4)
    assert rel.stats[0] == 0
    for rank in range(c.R):
        w = gen.weights(c, rank, W=64)
        a = oracle.pack(w, rank, g, p, c.R * c.n_slot)
        b = oracle.pack_relay(w, None, rank, g, p.slot_expert, rel.slot_src, c.R * c.n_slot)
        assert a[3] == b[3] == oracle.OK and a[2] == b[2]
        assert np.array_equal(a[1], b[1]) and np.array_equal(a[0][:a[2]], b[0][:b[2]])
