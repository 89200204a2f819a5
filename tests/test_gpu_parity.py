"""Parity of the HIP library with the oracle, byte for byte, on the same seeded
inputs: the five synthetic workloads at full size, every simulated rank of the
tiny workload, the adversarial fuzz corpus, error paths, determinism and
HIP-graph replay.  Needs an MI355X."""
import numpy as np
import pytest
import torch

import fuzz
import gen
import oracle
from invariants import check_plan

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    import gpu_path as gp
    import paper_2606_04101_amd as uep


def _workload(cid, m):
    c = gen.config(cid)
    g, og = gp.groups(c.R, c.E, c.n_slot, c.u_min, c.beta_num, c.beta_den)
    return c, g, og, gen.topk_all(c, m)


def _rstar(op, c):
    X = op.slot_expert
    outb = [int(((X >= 0) & (X // c.n_main == r)).sum()) for r in range(c.R)]
    return int(np.argmax(outb))


# ------------------------------------------------------------- count + plan

@pytest.mark.parametrize("cid,m", [(1, 0), (1, 3), (2, 0), (3, 0), (3, 7),
                                   (3, 15), (4, 0), (4, 1), (5, 0), (5, 57)])
def test_count_and_plan_workloads(cid, m):
    c, g, og, tk = _workload(cid, m)
    counts, st = gp.gpu_count(tk, c.E)
    ocounts, ost = oracle.count(tk, c.E, c.R)
    assert st == 0 and ost == 0
    assert np.array_equal(counts, ocounts)
    plan = gp.gpu_plan(ocounts, g)
    op = oracle.plan(ocounts, og)
    gp.assert_plan_equal(plan, op)
    check_plan(ocounts, og, op)


@pytest.mark.parametrize("cid,m", [(1, 1), (2, 3), (4, 2), (5, 9)])
def test_split_plan_entry_points(cid, m):
    """SolveReplication then SolveReroute through their own entry points give
    the same plan as ultraep_plan."""
    c, g, og, tk = _workload(cid, m)
    load, _ = oracle.count(tk, c.E, c.R)
    gp.assert_plan_equal(gp.gpu_plan(load, g, split=True), oracle.plan(load, og))


def test_qwen3_all_microbatches():
    c = gen.config(3)
    g, og = gp.groups(c.R, c.E, c.n_slot, c.u_min)
    for m in range(c.n_micro):
        tk = gen.topk_all(c, m)
        counts, st = gp.gpu_count(tk, c.E)
        assert st == 0
        gp.assert_plan_equal(gp.gpu_plan(counts, g), oracle.plan(counts, og))


def test_dsv3_prefill_all_layers_plan():
    c = gen.config(5)
    g, og = gp.groups(c.R, c.E, c.n_slot, c.u_min)
    for layer in range(c.n_micro):
        tk = gen.topk_all(c, layer)
        counts, st = gp.gpu_count(tk, c.E)
        assert st == 0
        gp.assert_plan_equal(gp.gpu_plan(counts, g), oracle.plan(counts, og))


# ------------------------------------------------------------- dispatch + pack

def _big_load(seed, R, E, base, hot, n_hot):
    rng = np.random.default_rng(seed)
    load = rng.integers(0, base, (R, E)).astype(np.int64)
    for e in rng.choice(E, n_hot, replace=False):
        load[:, e] += rng.integers(hot // 2, hot, R)
    assert load.sum() <= (1 << 30)
    return load.astype(np.int32)


@pytest.mark.parametrize("seed,R,E,NS,base,hot,n_hot", [
    (0, 8, 32, 2, 1 << 14, 1 << 20, 2),     # thresholds up to ~2^23: a long bisection
    (1, 16, 64, 1, 1 << 12, 1 << 21, 3),    # one slot, long bisection, total below 2^26
    (2, 8, 16, 3, 1 << 16, 1 << 23, 1),     # slack of 25 bits and more, total above 2^26
    (3, 4, 8, 2, 1 << 20, 1 << 25, 1),      # total near 2^30
    (4, 32, 128, 2, 1 << 10, 1 << 19, 4),   # several hosts per hot expert, large quotas
])
def test_plan_large_loads(seed, R, E, NS, base, hot, n_hot):
    """Load matrices far larger than any synthetic workload: bisections of
    more than 20 levels, slacks that need the wide probe, totals that need
    the 64-bit split.  The plan must still equal the oracle's."""
    load = _big_load(seed, R, E, base, hot, n_hot)
    g, og = gp.groups(R, E, NS, 1024)
    op = oracle.plan(load, og)
    gp.assert_plan_equal(gp.gpu_plan(load, g), op)
    gp.assert_plan_equal(gp.gpu_plan(load, g, split=True), op)
    check_plan(load, og, op)


def _many_transfers_load(seed):
    """64 ranks, 8 experts each, a seeded set of hot ranks whose every expert
    is heavy: the plans move 100-144 transfers, so the records of the best
    probe span two or three waves of 64."""
    rng = np.random.default_rng(seed)
    R, E = 64, 512
    NS = int(rng.choice([2, 3, 4]))
    u_min = int(rng.choice([1, 8, 64]))
    nm = E // R
    load = rng.integers(0, 50, (R, E))
    for h in rng.choice(R, int(rng.integers(8, 40)), replace=False):
        load[:, h * nm:(h + 1) * nm] += rng.integers(50, 400, (R, nm))
    return load.astype(np.int32), R, E, NS, u_min


@pytest.mark.parametrize("seed", [13, 15, 28, 31, 45, 52])
def test_plan_many_transfers(seed):
    """More than 64 accepted transfers: the round's record copy, the emit's
    record read, host positions and per-rank slot counts across waves of
    64 records, relay trees and the packing of the rank with the most
    outbound replicas, against the oracle."""
    load, R, E, NS, u_min = _many_transfers_load(seed)
    g, og = gp.groups(R, E, NS, u_min)
    op = oracle.plan(load, og)
    assert op.status == oracle.OK and op.stats[4] > 64
    gp.assert_plan_equal(gp.gpu_plan(load, g), op)
    gp.assert_plan_equal(gp.gpu_plan(load, g, split=True), op)
    check_plan(load, og, op)
    plan = gp.gpu_plan(load, g)
    rel = oracle.relay(og, op, 1)
    src = torch.empty(R * NS, dtype=torch.int32, device=gp.DEV)
    vol = torch.empty(R, dtype=torch.int32, device=gp.DEV)
    rst = torch.empty(4, dtype=torch.int64, device=gp.DEV)
    st = torch.zeros(1, dtype=torch.int32, device=gp.DEV)
    uep.ultraep_relay_plan(g, plan, 1, src, vol, rst, st)
    gp.assert_same("slot_src", src.cpu().numpy(), rel.slot_src.reshape(-1))
    X = op.slot_expert.reshape(R, NS)
    rank = int(np.argmax([((X >= 0) & (X // (E // R) == r)).sum() for r in range(R)]))
    rng = np.random.default_rng(seed)
    W = 1032
    w_h = rng.integers(0, 1 << 16, (E // R, W), dtype=np.uint16)
    ostg, odoff, n_out, ost = oracle.pack(w_h, rank, og, op, R * NS)
    assert ost == 0 and n_out > 0
    stg = torch.empty((n_out, W), dtype=torch.int16, device=gp.DEV)
    doff = torch.empty(R + 1, dtype=torch.int64, device=gp.DEV)
    uep.ultraep_pack_replicas(gp.dev_u16(w_h), W, rank, g, plan, stg, n_out, doff, st)
    gp.assert_same("staging", gp.host_u16(stg), ostg[:n_out])
    gp.assert_same("dest_off", doff.cpu().numpy(), odoff)
    assert int(st.item()) == 0


def test_tiny_every_rank():
    c, g, og, tk = _workload(1, 0)
    load, _ = oracle.count(tk, c.E, c.R)
    op = oracle.plan(load, og)
    plan = gp.gpu_plan(load, g)
    for r in range(c.R):
        x = gen.activations(c, 0, r)
        w = gen.weights(c, r)
        gp.check_rank(x, tk[r], w, r, g, og, plan, op)


@pytest.mark.parametrize("cid,m", [(2, 0), (3, 0), (4, 0), (5, 0)])
def test_full_size_dispatch_and_pack(cid, m):
    """Full-size rows (H) and expert blobs (W_e) for ranks 0, the rank with
    the most outbound replicas, and R-1."""
    c, g, og, tk = _workload(cid, m)
    load, _ = oracle.count(tk, c.E, c.R)
    op = oracle.plan(load, og)
    plan = gp.gpu_plan(load, g)
    rs = sorted({0, _rstar(op, c), c.R - 1})
    for r in rs:
        x = gen.activations(c, m, r)
        w = gen.weights(c, r) if r == rs[0] or r == _rstar(op, c) else None
        gp.check_rank(x, tk[r], w, r, g, og, plan, op, split=(r == rs[-1]))


@pytest.mark.parametrize("H", [520, 1032, 2056, 7176, 8192, 8200, 16400])
def test_scatter_row_widths(H):
    """Row widths for every register tiling of the scatter (16-byte chunks per
    lane 2, 4, 8, 16, and the multi-pass kernel above 8192 elements), with
    more tokens than the resident waves (each wave walks several tokens) and
    a quarter of the slots masked (zero-filled tail rows)."""
    R, E, NS, k, T = 4, 16, 2, 2, 2100
    g, og = gp.groups(R, E, NS, 8)
    rng = np.random.default_rng(H)
    tk = rng.integers(0, E, (R, T, k)).astype(np.int32)
    tk[rng.random((R, T, k)) < 0.25] = -1
    load, _ = oracle.count(tk, E, R)
    op = oracle.plan(load, og)
    plan = gp.gpu_plan(load, g)
    gp.assert_plan_equal(plan, op)
    r = 1
    x = rng.integers(0, 1 << 16, (T, H)).astype(np.uint16)
    gp.check_rank(x, tk[r], None, r, g, og, plan, op, split=True)


@pytest.mark.parametrize("H", [1032, 16400])
def test_scatter_routed_count_out_of_range(H):
    """The scatter reads the routed row count on the device: with the layout's
    own count the tail rows are zero-filled; a count below 0 or above T*k
    (not a layout of these slots) fills no row, and the routed rows are
    still the oracle's."""
    R, E, NS, k, T = 4, 16, 2, 2, 700
    g, og = gp.groups(R, E, NS, 8)
    rng = np.random.default_rng(H + 1)
    tk = rng.integers(0, E, (R, T, k)).astype(np.int32)
    tk[rng.random((R, T, k)) < 0.25] = -1
    load, _ = oracle.count(tk, E, R)
    op = oracle.plan(load, og)
    plan = gp.gpu_plan(load, g)
    r = 2
    x = rng.integers(0, 1 << 16, (T, H)).astype(np.uint16)
    osend, oros, oboff, ost = oracle.dispatch(x, tk[r], r, og, op)
    assert ost == 0
    V, nr = T * k, int(oboff[-1])
    assert 0 < nr < V
    _, ros, boff, st = gp.gpu_dispatch(x, tk[r], r, g, plan, split=True)
    assert st == 0 and np.array_equal(ros, oros) and np.array_equal(boff, oboff)
    ros_d = gp.dev_i32(ros)
    xd = gp.dev_u16(x)
    for count in (nr, -5, -(1 << 40), V + 3):
        send = torch.full((V, H), 0x5A5A, dtype=torch.int16, device=gp.DEV)
        n = torch.tensor([count], dtype=torch.int64, device=gp.DEV)
        print(f"scatter H={H} n_routed={count}", flush=True)
        uep.ultraep_dispatch_scatter(xd, T, k, H, ros_d, n, send)
        torch.cuda.synchronize()
        got = gp.host_u16(send)
        assert np.array_equal(got[:nr], osend[:nr]), f"routed rows differ (n_routed={count})"
        tail = np.zeros((V - nr, H), np.uint16) if count == nr else np.full((V - nr, H), 0x5A5A, np.uint16)
        assert np.array_equal(got[nr:], tail), f"tail rows (n_routed={count})"


@pytest.mark.parametrize("seed", range(0, 160))
def test_fuzz_parity(seed):
    case = fuzz.make_case(seed)
    g, og = gp.groups(case["R"], case["E"], case["n_slot"], case["u_min"],
                      case["beta_num"], case["beta_den"])
    tk = case["topk"]
    if tk.shape[1] > 0:
        counts, st = gp.gpu_count(tk, g.E)
        ocounts, _ = oracle.count(tk, g.E, g.R)
        assert st == 0 and np.array_equal(counts, ocounts)
    else:
        ocounts = np.zeros((g.R, g.E), np.int32)
    op = oracle.plan(ocounts, og)
    plan = gp.gpu_plan(ocounts, g)
    gp.assert_plan_equal(plan, op)
    rng = case["rng"]
    for r in sorted({0, g.R - 1}):
        x = rng.integers(0, 2 ** 16, (case["T"], case["H"])).astype(np.uint16)
        w = rng.integers(0, 2 ** 16, (g.n_main, case["W"])).astype(np.uint16)
        gp.check_rank(x, tk[r], w, r, g, og, plan, op, split=bool(seed % 2))


# ------------------------------------------------------------- error paths

@pytest.mark.parametrize("seed,W", [(0, 1 << 19), (1, 1 << 19), (2, 3 << 21), (3, 1 << 12)])
def test_pack_many_experts_and_tiles(seed, W):
    """Several replicated local experts with unequal fan-out and enough tiles
    to spread every expert over many workgroups: each (expert, tile) task
    must be copied exactly once, to every destination."""
    import types
    R, E, NS, rank = 16, 64, 4, 3
    g, og = gp.groups(R, E, NS, 1)
    rng = np.random.default_rng(seed)
    X = np.where(rng.random(R * NS) < 0.6,
                 rank * 4 + rng.integers(0, 4, R * NS),
                 rng.integers(-1, E, R * NS)).astype(np.int32)
    w = rng.integers(0, 1 << 16, (E // R, W), dtype=np.uint16)
    cap = R * NS
    ostg, odoff, n_out, ost = oracle.pack(w, rank, og, types.SimpleNamespace(slot_expert=X), cap)
    assert ost == 0 and n_out > 0
    plan = uep.Plan(g, gp.DEV)
    plan.slot_expert.copy_(torch.from_numpy(X))
    stg, doff, st = gp.gpu_pack(w, rank, g, plan, cap)
    assert st == 0
    assert np.array_equal(doff, odoff)
    assert np.array_equal(stg[:n_out], ostg[:n_out])
    assert (stg[n_out:] == 0x3C3C).all()


@pytest.mark.parametrize("cid,m,rank_pick", [(1, 0, "max"), (2, 0, "max"), (3, 5, "max"),
                                              (4, 0, "max"), (4, 0, "min"), (5, 11, "max")])
def test_reroute_and_pack(cid, m, rank_pick):
    """SolveReroute and the packing in one launch equal the oracle's plan and
    staging."""
    c, g, og, tk = _workload(cid, m)
    load, _ = oracle.count(tk, c.E, c.R)
    op = oracle.plan(load, og)
    outb = [int(((op.slot_expert >= 0) & (op.slot_expert // c.n_main == r)).sum()) for r in range(c.R)]
    rank = int(np.argmax(outb)) if rank_pick == "max" else int(np.argmin(outb))
    W = 8 * 4096 if cid > 1 else c.W
    w = gen.weights(c, rank, W=W)
    cap = c.R * c.n_slot
    ostg, odoff, n_out, ost = oracle.pack(w, rank, og, op, cap)
    plan = uep.Plan(g, gp.DEV)
    for f in uep.PLAN_FIELDS:
        getattr(plan, f).fill_(-12345)
    ld = gp.dev_i32(load)
    uep.ultraep_plan_replicate(ld, g, plan)
    st = gp.zero_status()
    stg = torch.full((cap, W), 0x3C3C, dtype=torch.int16, device=gp.DEV)
    doff = torch.full((c.R + 1,), -9, dtype=torch.int64, device=gp.DEV)
    uep.ultraep_reroute_and_pack(ld, g, plan, gp.dev_u16(w), W, rank, stg, cap, doff, st)
    torch.cuda.synchronize()
    assert int(st.item()) == 0
    gp.assert_plan_equal(plan, op)
    assert np.array_equal(doff.cpu().numpy(), odoff)
    s = gp.host_u16(stg)
    assert np.array_equal(s[:n_out], ostg[:n_out])
    assert (s[n_out:] == 0x3C3C).all()


def test_count_flags_bad_ids():
    tk = np.array([[[0, 3], [16, -1]], [[-2, 1], [2, 2]]], np.int32)
    counts, st = gp.gpu_count(tk, 16)
    assert st == uep.ULTRAEP_EDATA
    assert counts[0].tolist()[:4] == [1, 0, 0, 1] and counts[1].tolist()[:3] == [0, 1, 2]


@pytest.mark.parametrize("T,k,E,n_groups,bad", [(10001, 7, 96, 3, False), (8192, 8, 256, 2, False),
                                                 (4097, 8, 64, 1, True), (40000, 1, 1024, 2, False)])
def test_count_large_blocks(T, k, E, n_groups, bad):
    """Blocks above 32768 ids take the multi-workgroup path (unaligned sizes,
    masked slots, skewed ids, bad ids) and must equal the oracle."""
    rng = np.random.default_rng(T + E)
    hot = rng.integers(0, E, 4)
    tk = np.where(rng.random((n_groups, T, k)) < 0.5, hot[rng.integers(0, 4, (n_groups, T, k))],
                  rng.integers(-1, E, (n_groups, T, k))).astype(np.int32)
    if bad:
        tk[0, 17, 3] = E
        tk[0, 4000, 0] = -5
    counts, st = gp.gpu_count(tk, E)
    ocounts, ost = oracle.count(tk, E, n_groups)
    assert st == (uep.ULTRAEP_EDATA if bad else 0)
    assert np.array_equal(counts, ocounts)


def test_plan_flags_negative_load():
    g, og = gp.groups(4, 8, 1, 1)
    load = np.ones((4, 8), np.int32)
    load[2, 5] = -3
    plan = gp.gpu_plan(load, g)
    assert int(plan.stats[6].item()) == uep.ULTRAEP_EDATA


def test_dispatch_flags_plan_mismatch():
    g, og = gp.groups(4, 8, 1, 1)
    load = np.ones((4, 8), np.int32)
    plan = gp.gpu_plan(load, g)
    x = np.zeros((2, 8), np.uint16)
    _, _, _, st = gp.gpu_dispatch(x, np.array([[0, 1], [2, 3]], np.int32), 0, g, plan)
    assert st == uep.ULTRAEP_EDATA


@pytest.mark.parametrize("where,value", [(1, 1 << 30), (0, -5), (3, 1), (8, 1 << 20)])
def test_dispatch_flags_corrupt_host_lists(where, value):
    """A host list pointer array that is not a CSR of this group (an entry
    past the columns, a negative start, a decreasing pair, a total past the
    columns) raises ULTRAEP_EDATA; no row points outside send and no tail
    row is filled from the unwritten block offsets."""
    R, E, NS, k, T = 4, 8, 1, 2, 300
    g, og = gp.groups(R, E, NS, 1)
    rng = np.random.default_rng(where)
    tk = rng.integers(0, E, (R, T, k)).astype(np.int32)
    load, _ = oracle.count(tk, E, R)
    plan = gp.gpu_plan(load, g)
    hp = plan.host_ptr.cpu().numpy()
    hp[where] = value
    plan.host_ptr.copy_(torch.from_numpy(hp))
    x = rng.integers(0, 1 << 16, (T, 16)).astype(np.uint16)
    print(f"corrupt host_ptr[{where}] = {value}", flush=True)
    for split in (False, True):
        send, ros, boff, st = gp.gpu_dispatch(x, tk[0], 0, g, plan, split=split)
        assert st == uep.ULTRAEP_EDATA
        assert ((ros >= -1) & (ros < T * k)).all()
        assert (boff == -9).all()


def test_pack_flags_small_capacity():
    g, og = gp.groups(4, 8, 1, 1)
    load = np.zeros((4, 8), np.int32)
    load[0, 0] = 100
    op = oracle.plan(load, og)
    plan = gp.gpu_plan(load, g)
    n = int(op.stats[4])
    assert n >= 2
    w = np.arange(2 * 16, dtype=np.uint16).reshape(2, 16)
    stg, doff, st = gp.gpu_pack(w, 0, g, plan, n - 1)
    assert st == uep.ULTRAEP_ENOSPC
    _, odoff, _, _ = oracle.pack(w, 0, og, op, n)
    assert np.array_equal(doff, odoff)
    assert (stg == 0x3C3C).all()


def test_host_argument_errors_raise():
    g, _ = gp.groups(3, 8, 1, 1)  # E % R != 0
    with pytest.raises(uep.UltraEPError) as ei:
        uep.ultraep_plan_sizes(g)
    assert ei.value.code == uep.ULTRAEP_EINVAL


# ------------------------------------------------------------- determinism, graphs

def test_repeated_runs_identical():
    c, g, og, tk = _workload(4, 0)
    load, _ = oracle.count(tk, c.E, c.R)
    ref = gp.gpu_plan(load, g)
    ref_h = {f: getattr(ref, f).cpu().numpy() for f in uep.PLAN_FIELDS}
    for _ in range(20):
        p = gp.gpu_plan(load, g)
        for f in uep.PLAN_FIELDS:
            assert np.array_equal(getattr(p, f).cpu().numpy(), ref_h[f])
    r = 5
    x = gen.activations(c, 0, r)
    a = gp.gpu_dispatch(x, tk[r], r, g, ref)
    for _ in range(3):
        b = gp.gpu_dispatch(x, tk[r], r, g, ref, split=True)
        assert a[3] == b[3] == 0
        assert all(np.array_equal(u, v) for u, v in zip(a[:3], b[:3]))


@pytest.mark.parametrize("fork", [False, True])
def test_graph_replay_matches_eager(fork):
    """count -> plan -> dispatch -> pack captured in one HIP graph, replayed
    several times with eager work in between; every replay must equal the
    eager result.  fork: the pipeline the benchmark times, with the pack on a
    second stream after SolveReplication, alongside reroute and dispatch."""
    c, g, og, tk_all = _workload(1, 2)
    r = 2
    T, k, H = c.T, c.k, c.H
    W = 3 * c.H * 32
    x = gp.dev_u16(gen.activations(c, 2, r))
    w = gp.dev_u16(gen.weights(c, r, W=W))
    tk_all_d = gp.dev_i32(tk_all)
    tk_r = tk_all_d[r].contiguous()
    load = torch.empty((c.R, c.E), dtype=torch.int32, device=gp.DEV)
    st = gp.zero_status()
    plan = uep.Plan(g, gp.DEV)
    V = T * k
    send = torch.empty((V, H), dtype=torch.int16, device=gp.DEV)
    ros = torch.empty(V, dtype=torch.int32, device=gp.DEV)
    boff = torch.empty(c.R * g.S + 1, dtype=torch.int64, device=gp.DEV)
    ws = torch.empty(uep.ultraep_dispatch_ws_bytes(T, k, g), dtype=torch.uint8, device=gp.DEV)
    cap = c.R * c.n_slot
    stg = torch.zeros((cap, W), dtype=torch.int16, device=gp.DEV)
    doff = torch.empty(c.R + 1, dtype=torch.int64, device=gp.DEV)

    side = torch.cuda.Stream()

    def step():
        uep.ultraep_count(tk_all_d, T, k, c.E, c.R, load, st)
        if not fork:
            uep.ultraep_plan(load, g, plan)
            uep.ultraep_dispatch(x, tk_r, T, k, H, r, g, plan, send, ros, boff, ws, st)
            uep.ultraep_pack_replicas(w, W, r, g, plan, stg, cap, doff, st)
            return
        uep.ultraep_plan_replicate(load, g, plan)
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            uep.ultraep_pack_replicas(w, W, r, g, plan, stg, cap, doff, st)
        uep.ultraep_plan_reroute(load, g, plan)
        uep.ultraep_dispatch_layout(tk_r, T, k, r, g, plan, ros, boff, ws, st)
        uep.ultraep_dispatch_scatter(x, T, k, H, ros, boff[-1:], send)
        torch.cuda.current_stream().wait_stream(side)

    outs = lambda: [t.clone() for t in (load, send, ros, boff, stg, doff,
                                        *[getattr(plan, f) for f in uep.PLAN_FIELDS])]
    step()
    torch.cuda.synchronize()
    ref = outs()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        step()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    for i in range(4):
        for t in (load, send, ros, boff, doff, *[getattr(plan, f) for f in uep.PLAN_FIELDS]):
            t.fill_(-1)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        got = outs()
        for a, b in zip(got, ref):
            assert torch.equal(a, b), f"replay {i} differs"
        assert int(st.item()) == 0
