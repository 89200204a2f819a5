"""Pins of the oracle's two floating-point steps: the combine gather (the
reverse of the token assignment, weighted by the top-k gates) and the local
gradient reduction of replicated experts.  Their arithmetic is fp32 with a
fixed order (gates times bf16 rows summed over k ascending; main gradient
plus replicas in staging order), rounded to bf16 to nearest-even for the
combine.  Pinned by hand-computed fp32 and bf16 values where the order and
the rounding show, exact integer sums, and the fp64 definition within the
error bound of the arithmetic."""
import numpy as np
import pytest

import oracle


def bf16(x):
    """bf16 bit pattern of a float that bf16 represents exactly."""
    u = np.float32(x).view(np.uint32)
    assert u & 0xFFFF == 0, x
    return np.uint16(u >> 16)


def f32_of(b):
    return (np.asarray(b, np.uint16).astype(np.uint32) << 16).view(np.float32)


# ------------------------------------------------------------------ combine

def test_combine_unit_weight_k1_is_a_copy():
    rng = np.random.default_rng(0)
    y = (rng.standard_normal((40, 24)).astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
    ros = rng.permutation(40)[:30].astype(np.int32)
    out, st = oracle.combine(y, np.ones((30, 1), np.float32), ros)
    assert st == oracle.OK
    assert np.array_equal(out, y[ros])


@pytest.mark.parametrize("gate,want", [
    (1 + 2 ** -8, 0x3F80),            # exactly halfway between 1.0 and 1.0078125: even
    (1 + 3 * 2 ** -8, 0x3F82),        # halfway between 1.0078125 and 1.015625: even
    (1 + 2 ** -8 + 2 ** -20, 0x3F81),  # just above halfway: up
    (1 + 2 ** -8 - 2 ** -20, 0x3F80),  # just below halfway: down
    (-(1 + 3 * 2 ** -8), 0xBF82),     # sign kept
])
def test_combine_rounds_to_nearest_even(gate, want):
    y = np.array([[bf16(1.0)]], np.uint16)
    out, st = oracle.combine(y, np.array([[gate]], np.float32), np.array([0], np.int32))
    assert st == oracle.OK and int(out[0, 0]) == want


@pytest.mark.parametrize("order,want", [
    ((2.0 ** 25, 1.0, -2.0 ** 25), 0x0000),   # 2^25 + 1 rounds to 2^25 in fp32
    ((1.0, 2.0 ** 25, -2.0 ** 25), 0x0000),
    ((2.0 ** 25, -2.0 ** 25, 1.0), 0x3F80),   # cancellation first: exact
])
def test_combine_sums_in_fp32_in_k_order(order, want):
    """The exact sum is 1 in every order; fp32 in k order gives these."""
    y = np.array([[bf16(v)] for v in order], np.uint16)
    out, st = oracle.combine(y, np.ones((1, 3), np.float32), np.arange(3, dtype=np.int32))
    assert st == oracle.OK and int(out[0, 0]) == want


def test_combine_skips_masked_slots():
    y = np.array([[bf16(2.0)], [bf16(8.0)]], np.uint16)
    gate = np.array([[0.5, 0.25], [0.75, 0.5]], np.float32)
    ros = np.array([1, -1, -1, -1], np.int32)
    out, st = oracle.combine(y, gate, ros)
    assert st == oracle.OK
    assert out[:, 0].tolist() == [bf16(4.0), 0x0000]   # 0.5*8; no routed slot: +0


def test_combine_rejects_rows_out_of_range():
    y = np.zeros((4, 8), np.uint16)
    assert oracle.combine(y, np.ones((2, 2), np.float32), np.array([0, 1, 2, 4], np.int32))[1] == oracle.EDATA
    assert oracle.combine(y, np.ones((2, 2), np.float32), np.array([0, 1, -2, 3], np.int32))[1] == oracle.EDATA


@pytest.mark.parametrize("seed,k", [(0, 8), (1, 2), (2, 5)])
def test_combine_within_error_bound_of_the_fp64_definition(seed, k):
    """|out - S| <= 2^-8 |S| + 4 k 2^-24 sum|g y| for S the exact weighted
    sum (fp64): k fp32 products and sums, then one bf16 rounding."""
    rng = np.random.default_rng(seed)
    T, H = 64, 96
    yf = rng.standard_normal((T * k, H)).astype(np.float32)
    y = (yf.view(np.uint32) >> 16).astype(np.uint16)
    z = rng.standard_normal((T, k))
    gate = (np.exp(z) / np.exp(z).sum(1, keepdims=True)).astype(np.float32)
    ros = rng.permutation(T * k).astype(np.int32)
    ros[rng.random(T * k) < 0.1] = -1
    out, st = oracle.combine(y, gate, ros)
    assert st == oracle.OK
    yv = f32_of(y).astype(np.float64)
    r = ros.reshape(T, k)
    terms = np.where((r >= 0)[:, :, None], gate.astype(np.float64)[:, :, None] * yv[np.maximum(r, 0)], 0.0)
    S = terms.sum(1)
    bound = 2.0 ** -8 * np.abs(S) + 4 * k * 2.0 ** -24 * np.abs(terms).sum(1) + 1e-30
    assert np.all(np.abs(f32_of(out).astype(np.float64) - S) <= bound)


# ------------------------------------------------------------------ gradient reduction

def _group_one_main():
    return oracle.Group(4, 4, 2, 1)   # one main expert per rank, two slots


def test_grad_reduce_integer_sums_are_exact():
    g = _group_one_main()
    X = np.array([[-1, -1], [0, 2], [0, 3], [1, 0]], np.int32)  # rank 0's expert 0 on (1,0) (2,0) (3,1)
    rng = np.random.default_rng(3)
    W = 16
    main = rng.integers(-1000, 1000, (1, W)).astype(np.float32)
    rg = rng.integers(-1000, 1000, (3, W)).astype(np.float32)
    mg2, rg2, n, st = oracle.grad_reduce(main, rg, 0, g, X, 8)
    assert st == oracle.OK and n == 3
    assert np.array_equal(mg2[0], main[0] + rg.sum(0))
    assert not rg2.any()


def test_grad_reduce_fp32_sequential_from_the_main_value():
    """2^24 + 1 + 1 in fp32 is 2^24 (each +1 is a tie that rounds to even),
    although 2^24 + 2 is representable; 1 + 2^24 - 2^24 is 0."""
    g = _group_one_main()
    X = np.array([[-1, -1], [0, -1], [0, -1], [-1, -1]], np.int32)
    main = np.array([[2.0 ** 24, 1.0]], np.float32)
    rg = np.array([[1.0, 2.0 ** 24], [1.0, -2.0 ** 24]], np.float32)
    mg2, rg2, n, st = oracle.grad_reduce(main, rg, 0, g, X, 2)
    assert st == oracle.OK and n == 2
    assert mg2[0].tolist() == [2.0 ** 24, 0.0]


def test_grad_reduce_follows_staging_order():
    """Expert 0 sits on (2, 0) and (1, 1): staging order is rank 1's slot
    first.  main 1, (1,1): 2^24, (2,0): -2^24 gives 0 in that order (1 the
    other way)."""
    g = _group_one_main()
    X = np.array([[-1, -1], [3, 0], [0, -1], [-1, -1]], np.int32)
    main = np.array([[1.0]], np.float32)
    rg = np.array([[2.0 ** 24], [-2.0 ** 24]], np.float32)   # staging order
    mg2, _, n, st = oracle.grad_reduce(main, rg, 0, g, X, 2)
    assert st == oracle.OK and n == 2 and mg2[0, 0] == 0.0


def test_grad_reduce_entries_map_to_experts_in_staging_order():
    """Rank 0's expert 0 sits on (1, 1) and expert 1 on (2, 0): in staging
    order (destination rank first) entry 0 is expert 0's replica."""
    g = oracle.Group(4, 8, 2, 1)
    X = np.array([[-1, -1], [-1, 0], [1, -1], [-1, -1]], np.int32)
    main = np.zeros((2, 1), np.float32)
    rg = np.array([[5.0], [7.0]], np.float32)
    mg2, _, n, st = oracle.grad_reduce(main, rg, 0, g, X, 2)
    assert st == oracle.OK and n == 2 and mg2[:, 0].tolist() == [5.0, 7.0]


def test_grad_reduce_untouched_without_replicas_and_capacity():
    g = _group_one_main()
    X = np.array([[-1, -1], [2, -1], [3, -1], [1, -1]], np.int32)  # nothing of rank 0
    main = np.full((1, 4), 7.5, np.float32)
    mg2, _, n, st = oracle.grad_reduce(main, np.zeros((0, 4), np.float32), 0, g, X, 0)
    assert st == oracle.OK and n == 0 and np.array_equal(mg2, main)
    X = np.array([[-1, -1], [0, -1], [0, -1], [0, -1]], np.int32)
    rg = np.ones((3, 4), np.float32)
    mg2, rg2, n, st = oracle.grad_reduce(main, rg, 0, g, X, 2)
    assert st == oracle.ENOSPC and n == 3
    assert np.array_equal(mg2, main) and np.array_equal(rg2, rg)


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_grad_reduce_within_error_bound_of_the_fp64_sum(seed):
    """Several local experts with unequal fan-out: each main gradient is
    within (f + 1) 2^-24 sum|terms| of its fp64 sum; replicas zeroed."""
    rng = np.random.default_rng(seed)
    R, E, NS, rank = 8, 32, 3, 2
    g = oracle.Group(R, E, NS, 1)
    nm = E // R
    X = np.where(rng.random((R, NS)) < 0.6, rank * nm + rng.integers(0, nm, (R, NS)),
                 rng.integers(-1, E, (R, NS))).astype(np.int32)
    for t in range(R):  # one copy of an expert per rank, none on its home
        seen = set()
        for s in range(NS):
            e = X[t, s]
            if e >= 0 and (e // nm == t or e in seen):
                X[t, s] = -1
            elif e >= 0:
                seen.add(e)
    W = 64
    main = rng.standard_normal((nm, W)).astype(np.float32)
    ent = [(t, s) for t in range(R) for s in range(NS) if X[t, s] >= 0 and X[t, s] // nm == rank]
    rg = rng.standard_normal((len(ent), W)).astype(np.float32) * 100
    mg2, rg2, n, st = oracle.grad_reduce(main, rg, rank, g, X, R * NS)
    assert st == oracle.OK and n == len(ent) and not rg2.any()
    for l in range(nm):
        idx = [i for i, (t, s) in enumerate(ent) if X[t, s] == rank * nm + l]
        terms = np.vstack([main[l:l + 1].astype(np.float64)] + [rg[i:i + 1].astype(np.float64) for i in idx])
        S = terms.sum(0)
        bound = (len(idx) + 1) * 2.0 ** -24 * np.abs(terms).sum(0)
        assert np.all(np.abs(mg2[l].astype(np.float64) - S) <= bound)
        if not idx:
            assert np.array_equal(mg2[l], main[l])
