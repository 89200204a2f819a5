"""The bound behind SolveReroute's small-demand chain (Sec. 5.2, the split
of a source's residual demand by largest remainder): with c = (lh / D) *
(1 - 2^-20) rounded to fp32 and y = fl32(c * u), trunc(y) is floor(lh * u /
D) or one less whenever 1 <= lh <= D < 2^19 and 0 <= u <= D, so the
remainder lh * u - trunc(y) * D lies in [0, 2D).  The GPU kernel relies on
it to take the floor and the remainder with one subtraction and a min.
Emulated here with numpy's IEEE fp32 (round to nearest even, as the
kernel's v_mul_f32 and fp64-to-fp32 conversion; v_cvt_i32_f32 truncates)
over random and worst-case inputs.  CPU only."""
import math

import numpy as np
import pytest

LIMIT = 1 << 19


def estimate(lh, u, D):
    c = (lh.astype(np.float64) * (1.0 - 2.0 ** -20) / D.astype(np.float64)).astype(np.float32)
    y = c * u.astype(np.float32)
    assert y.dtype == np.float32
    return np.trunc(y).astype(np.int64)


def check(lh, u, D):
    lh, u, D = (np.asarray(v, np.int64) for v in (lh, u, D))
    assert (1 <= lh).all() and (lh <= D).all() and (D < LIMIT).all()
    assert (0 <= u).all() and (u <= D).all()
    be = estimate(lh, u, D)
    fl = (lh * u) // D
    bad = ~((be == fl) | (be == fl - 1))
    assert not bad.any(), list(zip(lh[bad][:5], u[bad][:5], D[bad][:5], be[bad][:5], fl[bad][:5]))
    re = lh * u - be * D
    assert ((re >= 0) & (re < 2 * D)).all()


@pytest.mark.parametrize("seed", range(4))
def test_random(seed):
    rng = np.random.default_rng(seed)
    n = 1 << 20
    D = rng.integers(1, LIMIT, n)
    lh = rng.integers(1, D + 1)
    u = rng.integers(0, D + 1)
    check(lh, u, D)


def test_near_the_limit():
    # the largest demands and quotas, where the estimate's absolute error is
    # largest, and quotients that are exact integers (the estimate falls
    # just below them)
    rng = np.random.default_rng(7)
    n = 1 << 20
    D = rng.integers(LIMIT - 4096, LIMIT, n)
    lh = D - rng.integers(0, 64, n)
    u = D - rng.integers(0, 64, n)
    check(lh, u, D)
    check(D, u, D)          # lh = D: the quotient is u itself
    check(lh, D, D)         # u = D: the quotient is lh
    k = rng.integers(1, 512, n)
    Dk = (LIMIT - 1) // k * k
    check(np.minimum(Dk, (LIMIT - 1) // 2), Dk // k * rng.integers(1, k + 1), Dk)


def test_quotients_just_below_an_integer():
    # lh * u = k * D - 1: the quotient sits 1/D below an integer, where an
    # unbiased fp32 estimate rounds up to it (one above the floor); the
    # 2^-20 bias keeps the estimate below
    rng = np.random.default_rng(11)
    rows = []
    while len(rows) < 20000:
        D = int(rng.integers(LIMIT // 2, LIMIT))
        lh = int(rng.integers(1, D + 1))
        if math.gcd(lh, D) == 1:
            rows.append((lh, (D - 1) * pow(lh, -1, D) % D, D))
    lh, u, D = np.array(rows, np.int64).T
    assert (((lh * u) % D) == D - 1).all()
    check(lh, u, D)


def test_exhaustive_small():
    # every (lh, u) for a few D, the small end of the range
    for D in (1, 2, 3, 7, 64, 255, 1000):
        lh, u = np.meshgrid(np.arange(1, D + 1), np.arange(0, D + 1), indexing="ij")
        check(lh.ravel(), u.ravel(), np.full(lh.size, D))
