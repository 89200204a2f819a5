"""Parity of ultraep_combine and ultraep_grad_reduce with the oracle, bit for
bit: both follow one fixed fp32 order (gates times rows over k ascending;
main gradient plus replicas in staging order), so the outputs are equal
patterns.  NaN results of the fp32 reduction are compared as NaN only (their
payload depends on the processor).  Needs an MI355X."""
import numpy as np
import pytest
import torch

import gen
import oracle
from test_gpu_relay import dense_slot_map, plan_on_device
from test_oracle_relay import csr_from_slots

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    import gpu_path as gp
    import paper_2606_04101_amd as uep


def bf16_normals(rng, shape):
    """Finite bf16 patterns of magnitude in [2^-3, 2^5), either sign, any
    mantissa (drawn as 16-bit integers: fast at the prefill size)."""
    u = rng.integers(0, 1 << 16, shape, dtype=np.uint16)
    return ((u & 0x807F) | ((0x7C + ((u >> 7) & 0x7)) << 7)).astype(np.uint16)


def softmax_gates(rng, T, k):
    z = rng.standard_normal((T, k))
    return (np.exp(z) / np.exp(z).sum(1, keepdims=True)).astype(np.float32)


def gpu_combine(y, gate, ros, H):
    T, k = gate.shape
    out = torch.full((max(T, 1), H), 0x5A5A, dtype=torch.int16, device=gp.DEV)
    st = gp.zero_status()
    uep.ultraep_combine(gp.dev_u16(y) if y.size else None, y.shape[0],
                        torch.from_numpy(np.ascontiguousarray(gate)).to(gp.DEV),
                        gp.dev_i32(ros.reshape(-1)), T, k, H, out, st)
    torch.cuda.synchronize()
    return gp.host_u16(out)[:T], int(st.item())


def check_combine(y, gate, ros, sample=None):
    T, k = gate.shape
    H = y.shape[1]
    out, st = gpu_combine(y, gate, ros, H)
    assert st == 0
    if sample is None:
        o, ost = oracle.combine(y, gate, ros)
        assert ost == oracle.OK
        assert np.array_equal(out, o)
    else:  # the oracle on a sample of tokens
        r = ros.reshape(T, k)
        o, ost = oracle.combine(y, gate[sample], r[sample])
        assert ost == oracle.OK
        assert np.array_equal(out[sample], o)


@pytest.mark.parametrize("cid", [1, 2, 3, 4, 5])
def test_combine_workloads(cid):
    """Rows in the dispatch layout of the rank with the most replicas,
    every row of y a bf16 normal, softmax gates; the prefill-sized
    workload is checked on 2048 sampled tokens."""
    c = gen.config(cid)
    g, og = gp.groups(c.R, c.E, c.n_slot, c.u_min, c.beta_num, c.beta_den)
    tk = gen.topk_all(c, 0)
    load, _ = oracle.count(tk, c.E, c.R)
    op = oracle.plan(load, og)
    X = op.slot_expert
    rank = int(np.argmax([((X >= 0) & (X // c.n_main == r)).sum() for r in range(c.R)]))
    plan = gp.gpu_plan(load, g)
    x = np.zeros((c.T, 8), np.uint16)  # the layout does not depend on H
    _, ros, _, st = gp.gpu_dispatch(x, tk[rank], rank, g, plan)
    assert st == 0
    rng = np.random.default_rng(cid)
    V = c.T * c.k
    y = bf16_normals(rng, (V, c.H))
    gate = softmax_gates(rng, c.T, c.k)
    sample = None if cid < 5 else np.sort(rng.choice(c.T, 2048, replace=False))
    check_combine(y, gate, ros.reshape(c.T, c.k), sample)


@pytest.mark.parametrize("T,k,H", [(1, 1, 8), (7, 3, 136), (300, 8, 520), (129, 12, 64),
                                   (64, 64, 16), (2100, 8, 7176), (5, 16, 8200), (0, 8, 64)])
def test_combine_shapes(T, k, H):
    """Ragged row widths, k above the eight rows loaded together, more
    tokens than resident waves, a quarter of the slots masked, T = 0."""
    rng = np.random.default_rng(T * 1000 + k * 10 + H)
    n_rows = T * k + 5
    y = bf16_normals(rng, (n_rows, H))
    gate = softmax_gates(rng, T, k) if T else np.zeros((0, k), np.float32)
    ros = rng.permutation(n_rows)[:T * k].astype(np.int32)
    ros[rng.random(T * k) < 0.25] = -1
    if T == 0:
        out, st = gpu_combine(y, gate, ros, H)
        assert st == 0
        return
    check_combine(y, gate, ros.reshape(T, k))


def test_combine_special_values():
    """Signed zeros, infinities, NaNs, subnormal rows and subnormal
    products, large values that overflow to infinity, negative gates."""
    rng = np.random.default_rng(11)
    T, k, H = 512, 4, 64
    specials = np.array([0x0000, 0x8000, 0x7F80, 0xFF80, 0x7FC0, 0xFFC1, 0x0001, 0x807F,
                         0x0080, 0x7F7F, 0xFF7F, 0x3F80, 0xBF80, 0x4C00, 0xCC00], np.uint16)
    y = rng.choice(specials, (T * k, H)).astype(np.uint16)
    gate = rng.choice(np.array([1.0, -0.5, 0.0, -0.0, 2.0 ** -100, 3.0e38, 0.25], np.float32),
                      (T, k)).astype(np.float32)
    ros = rng.permutation(T * k).astype(np.int32)
    check_combine(y, gate, ros.reshape(T, k))


def test_combine_flags_rows_out_of_range():
    rng = np.random.default_rng(2)
    y = bf16_normals(rng, (16, 64))
    gate = softmax_gates(rng, 4, 4)
    ros = np.arange(16, dtype=np.int32)
    ros[5] = 16
    assert gpu_combine(y, gate, ros, 64)[1] == uep.ULTRAEP_EDATA


# ------------------------------------------------------------------ gradient reduction

def gpu_grad_reduce(main, rg, rank, g, plan, cap):
    W = main.shape[1]
    mg = torch.from_numpy(np.ascontiguousarray(main, np.float32)).to(gp.DEV)
    rgd = torch.zeros((max(cap, 1), W), dtype=torch.float32, device=gp.DEV)
    if rg.shape[0]:
        rgd[:rg.shape[0]] = torch.from_numpy(np.ascontiguousarray(rg, np.float32))
    st = gp.zero_status()
    uep.ultraep_grad_reduce(mg, rgd, W, rank, g, plan, cap, st)
    torch.cuda.synchronize()
    return mg.cpu().numpy(), rgd.cpu().numpy()[:rg.shape[0]], int(st.item())


def same_f32(a, b):
    """Equal bit patterns, NaNs compared as NaN."""
    na, nb = np.isnan(a), np.isnan(b)
    return np.array_equal(na, nb) and np.array_equal(a.view(np.uint32)[~na], b.view(np.uint32)[~nb])


def check_reduce(g, og, plan, X, rank, W, rng, special=False):
    nm = g.n_main
    Xr = np.asarray(X).reshape(g.R, g.n_slot)
    n = int(((Xr >= 0) & (Xr // nm == rank)).sum())
    if special:
        vals = np.array([0.0, -0.0, 1.0, -1.0, 2.0 ** 24, -2.0 ** 24, 1e-45, -1e-45, 3e38, -3e38,
                         np.inf, -np.inf, 1.5, 2.0 ** -126], np.float32)
        main = rng.choice(vals, (nm, W)).astype(np.float32)
        rg = rng.choice(vals, (n, W)).astype(np.float32)
    else:
        main = rng.standard_normal((nm, W)).astype(np.float32)
        rg = (rng.standard_normal((n, W)) * 10).astype(np.float32)
    cap = g.R * g.n_slot
    omg, org, on, ost = oracle.grad_reduce(main, rg, rank, og, X, cap)
    assert ost == oracle.OK and on == n
    mg, rgo, st = gpu_grad_reduce(main, rg, rank, g, plan, cap)
    assert st == 0
    assert same_f32(mg, omg), f"main_grad rank {rank}"
    assert same_f32(rgo, org), f"replicas not cleared rank {rank}"
    return n


@pytest.mark.parametrize("cid", [1, 2, 3, 4, 5])
def test_grad_reduce_workloads(cid):
    c = gen.config(cid)
    g, og = gp.groups(c.R, c.E, c.n_slot, c.u_min, c.beta_num, c.beta_den)
    load, _ = oracle.count(gen.topk_all(c, 0), c.E, c.R)
    op = oracle.plan(load, og)
    plan = gp.gpu_plan(load, g)
    rng = np.random.default_rng(cid)
    X = op.slot_expert
    outb = [int(((X >= 0) & (X // c.n_main == r)).sum()) for r in range(c.R)]
    for rank in sorted({0, int(np.argmax(outb)), c.R - 1}):
        check_reduce(g, og, plan, X, rank, 8 * 4100, rng)


@pytest.mark.parametrize("seed,R,E,NS,n_hot,W", [(0, 64, 64, 4, 5, 4100), (1, 64, 256, 4, 12, 1 << 14),
                                                 (4, 16, 1024, 16, 30, 4), (5, 64, 128, 4, 40, 12)])
def test_grad_reduce_dense_slot_maps(seed, R, E, NS, n_hot, W):
    """Fan-outs up to 63 replicas per expert, several replicated experts per
    rank, ragged blob sizes; every rank."""
    g, og = gp.groups(R, E, NS, 1)
    p = csr_from_slots(R, E, NS, dense_slot_map(seed, R, E, NS, n_hot))
    plan = plan_on_device(g, p)
    rng = np.random.default_rng(seed)
    tot = sum(check_reduce(g, og, plan, p.slot_expert, rank, W, rng) for rank in range(R))
    assert tot == int((np.asarray(p.slot_expert) >= 0).sum())


def test_grad_reduce_special_values():
    g, og = gp.groups(64, 64, 4, 1)
    p = csr_from_slots(64, 64, 4, dense_slot_map(0, 64, 64, 4, 5))
    plan = plan_on_device(g, p)
    rng = np.random.default_rng(9)
    for rank in range(0, 64, 7):
        check_reduce(g, og, plan, p.slot_expert, rank, 1024, rng, special=True)


def test_grad_reduce_full_size_blob():
    """One replicated expert of the DeepSeek-V3-shaped layer at its full
    blob size (3 * 7168 * 2048 fp32 gradients)."""
    c = gen.config(4)
    g, og = gp.groups(c.R, c.E, c.n_slot, c.u_min, c.beta_num, c.beta_den)
    load, _ = oracle.count(gen.topk_all(c, 0), c.E, c.R)
    op = oracle.plan(load, og)
    plan = gp.gpu_plan(load, g)
    X = op.slot_expert
    rank = int(np.argmax([((X >= 0) & (X // c.n_main == r)).sum() for r in range(c.R)]))
    assert check_reduce(g, og, plan, X, rank, c.W, np.random.default_rng(4)) > 0


def test_grad_reduce_capacity():
    g, og = gp.groups(4, 4, 2, 1)
    X = np.array([[-1, -1], [0, -1], [0, -1], [0, -1]], np.int32)
    plan = plan_on_device(g, csr_from_slots(4, 4, 2, X))
    main = np.ones((1, 8), np.float32)
    mg = torch.from_numpy(main).to(gp.DEV)
    rg = torch.ones((2, 8), dtype=torch.float32, device=gp.DEV)
    st = gp.zero_status()
    uep.ultraep_grad_reduce(mg, rg, 8, 0, g, plan, 2, st)
    torch.cuda.synchronize()
    assert int(st.item()) == uep.ULTRAEP_ENOSPC
    assert (mg.cpu().numpy() == 1).all() and (rg.cpu().numpy() == 1).all()


def test_graph_replay_of_relay_combine_reduce():
    """ultraep_relay_plan, ultraep_pack_relay, ultraep_combine and
    ultraep_grad_reduce captured in one HIP graph after count, plan and
    dispatch, replayed several times with the outputs poisoned and the
    gradient inputs restored between replays; every replay equals the eager
    result."""
    c = gen.config(3)
    g, og = gp.groups(c.R, c.E, c.n_slot, c.u_min, c.beta_num, c.beta_den)
    tk_all = gen.topk_all(c, 0)
    load0, _ = oracle.count(tk_all, c.E, c.R)
    op = oracle.plan(load0, og)
    X = op.slot_expert
    r = int(np.argmax([((X >= 0) & (X // c.n_main == q)).sum() for q in range(c.R)]))
    T, k, H = 512, c.k, 256          # combine over 512 tokens of narrow rows
    W = 8 * 256
    rng = np.random.default_rng(21)
    dev = gp.DEV
    tk_all_d = gp.dev_i32(tk_all)
    load = torch.empty((c.R, c.E), dtype=torch.int32, device=dev)
    st = gp.zero_status()
    plan = uep.Plan(g, dev)
    V = T * k
    send = torch.empty((V, H), dtype=torch.int16, device=dev)
    ros = torch.empty(V, dtype=torch.int32, device=dev)
    gate = torch.from_numpy(softmax_gates(rng, T, k)).to(dev)
    out = torch.empty((T, H), dtype=torch.int16, device=dev)
    src = torch.empty(c.R * c.n_slot, dtype=torch.int32, device=dev)
    vol = torch.empty(c.R, dtype=torch.int32, device=dev)
    rst = torch.empty(4, dtype=torch.int64, device=dev)
    cap = c.R * c.n_slot
    w = gp.dev_u16(rng.integers(0, 1 << 16, (c.n_main, W), dtype=np.uint16))
    rsrc = gp.dev_u16(rng.integers(0, 1 << 16, (c.n_slot, W), dtype=np.uint16))
    stg = torch.zeros((cap, W), dtype=torch.int16, device=dev)
    doff = torch.empty(c.R + 1, dtype=torch.int64, device=dev)
    mg0 = torch.from_numpy(rng.standard_normal((c.n_main, 64)).astype(np.float32)).to(dev)
    rg0 = torch.from_numpy(rng.standard_normal((cap, 64)).astype(np.float32)).to(dev)
    mg, rg = mg0.clone(), rg0.clone()

    def step():
        uep.ultraep_count(tk_all_d, c.T, k, c.E, c.R, load, st)
        uep.ultraep_plan(load, g, plan)
        uep.ultraep_relay_plan(g, plan, 1, src, vol, rst, st)
        uep.ultraep_pack_relay(w, rsrc, W, r, g, plan, src, stg, cap, doff, st)
        uep.ultraep_grad_reduce(mg, rg, 64, r, g, plan, cap, st)
        uep.ultraep_combine(send, V, gate, ros, T, k, H, out, st)

    # a fixed layout for the combine: rows in slot order, every 7th masked
    ros.copy_(torch.arange(V, dtype=torch.int32, device=dev))
    ros[::7] = -1
    send.copy_(torch.from_numpy(bf16_normals(rng, (V, H)).view(np.int16)).to(dev))
    outs = lambda: [t.clone() for t in (load, src, vol, rst, stg, doff, mg, rg, out,
                                        *[getattr(plan, f) for f in uep.PLAN_FIELDS])]
    step()
    torch.cuda.synchronize()
    assert int(st.item()) == 0
    ref = outs()
    mg.copy_(mg0)
    rg.copy_(rg0)
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
        for t in (load, src, vol, rst, doff, out, *[getattr(plan, f) for f in uep.PLAN_FIELDS]):
            t.fill_(-1)
        mg.copy_(mg0)
        rg.copy_(rg0)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for a, b in zip(outs(), ref):
            assert torch.equal(a, b), f"replay {i} differs"
        assert int(st.item()) == 0
