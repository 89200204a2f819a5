"""Seeded corpus of small adversarial cases shared by the oracle tests and the
GPU parity tests.  Pure input generation: no balancing arithmetic here."""
from __future__ import annotations

import numpy as np

PATTERNS = ("random", "hot", "zero", "balanced", "masked", "dup", "zipf",
            "two_hot")


def make_case(seed: int):
    rng = np.random.default_rng(10_000 + seed)
    R = int(rng.integers(1, 9))
    nm = int(rng.integers(1, 5))
    E = R * nm
    NS = int(rng.integers(0, 4))
    k = int(rng.integers(1, min(4, E) + 1))
    T = int(rng.choice([0, 1, 7, 64, 129, 300]))
    u_min = int(rng.choice([1, 2, 7, 32]))
    beta = [(101, 100), (100, 100), (3, 2)][int(rng.integers(0, 3))]
    pat = PATTERNS[seed % len(PATTERNS)]
    V = T * k
    tk = np.empty((R, V), np.int32)
    for r in range(R):
        if pat == "random":
            tk[r] = rng.integers(0, E, V)
        elif pat == "hot":
            tk[r] = 0 if r % 2 == 0 else rng.integers(0, E, V)
        elif pat == "zero":
            tk[r] = -1
        elif pat == "balanced":
            tk[r] = np.arange(V) % E
        elif pat == "masked":
            v = rng.integers(0, E, V)
            v[rng.random(V) < 0.25] = -1
            tk[r] = v
        elif pat == "dup":
            tk[r] = rng.integers(0, max(1, E // 2), V)
        elif pat == "zipf":
            w = 1.0 / np.arange(1, E + 1) ** 1.3
            tk[r] = rng.choice(E, V, p=w / w.sum())
        elif pat == "two_hot":
            tk[r] = rng.choice([0, E - 1], V) if E > 1 else 0
    topk = tk.reshape(R, T, k)
    H = int(rng.choice([8, 64, 136]))
    W = int(rng.choice([8, 256, 4104]))
    return dict(seed=seed, pattern=pat, R=R, E=E, n_slot=NS, k=k, T=T,
                u_min=u_min, beta_num=beta[0], beta_den=beta[1], topk=topk,
                H=H, W=W, rng=rng)


def corpus(n: int = 160):
    return [make_case(s) for s in range(n)]
