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


MID_PATTERNS = ("zipf", "masked_zipf", "uniform", "hot_ranks", "one_expert")


def make_mid_case(seed: int):
    """Groups between the small corpus and the full workloads: any rank count
    up to 64 (not only powers of two), up to 1024 experts and 256 redundant
    slots, top-k up to 64, blocks of more than 32768 ids, rows wider than
    8192 elements and ragged blob widths."""
    rng = np.random.default_rng(20_000 + seed)
    R = int(rng.choice([2, 3, 5, 8, 12, 16, 24, 32, 48, 64]))
    nm = int(rng.integers(1, min(16, 1024 // R) + 1))
    E = R * nm
    NS = int(rng.integers(0, min(4, 256 // R) + 1))
    ks = [v for v in (1, 2, 4, 6, 8, 12, 16, 64) if v <= E]
    k = int(rng.choice(ks))
    H = int(rng.choice([8, 72, 1032, 7168, 8200, 12296]))
    # at most 2^25 send elements (64 MiB) and 72000 ids per rank
    vmax = min(72000, (1 << 25) // H)
    T = int(rng.choice([0, 1, int(2 + (vmax // k - 1) * rng.random() ** 0.5)], p=[0.05, 0.05, 0.9]))
    # u_min from 1 up to the mean expert load, so that most cases replicate
    lam_mean = R * T * k / E
    u_min = max(1, int(lam_mean * float(rng.choice([0.0, 0.02, 0.1, 0.5, 1.0]))))
    beta = [(101, 100), (1, 1), (5, 4)][int(rng.integers(0, 3))]
    pat = MID_PATTERNS[seed % len(MID_PATTERNS)]
    V = T * k
    alpha = float(rng.uniform(0.5, 1.5))
    pz = 1.0 / np.arange(1, E + 1) ** alpha
    pz = pz[rng.permutation(E)]
    pz /= pz.sum()
    tk = np.empty((R, V), np.int32)
    for r in range(R):
        if pat == "zipf":
            tk[r] = rng.choice(E, V, p=pz)
        elif pat == "masked_zipf":
            v = rng.choice(E, V, p=pz)
            v[rng.random(V) < 0.2] = -1
            tk[r] = v
        elif pat == "uniform":
            tk[r] = rng.integers(0, E, V)
        elif pat == "hot_ranks":  # the experts of a few ranks draw most ids
            hot = rng.choice(R, max(1, R // 8), replace=False)
            w = np.ones(E)
            for h in hot:
                w[h * nm:(h + 1) * nm] = 40.0
            tk[r] = rng.choice(E, V, p=w / w.sum())
        elif pat == "one_expert":  # one expert takes half of every rank's ids
            v = rng.integers(0, E, V)
            v[rng.random(V) < 0.5] = seed % E
            tk[r] = v
    W = int(8 * rng.integers(1, 8193))
    return dict(seed=seed, pattern=pat, R=R, E=E, n_slot=NS, k=k, T=T,
                u_min=u_min, beta_num=beta[0], beta_den=beta[1],
                topk=tk.reshape(R, T, k), H=H, W=W, rng=rng)
