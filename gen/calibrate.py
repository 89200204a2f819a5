"""Calibrate the Zipf bias scale c of the skewed workloads and freeze it.

For each Zipf workload, c is found by bisection on [0, c_max] so that
microbatch 0 has the target max/mean rank load (2.0 for the GLM-4.5-Air
shaped layer, 3.5 for the DeepSeek-V3 training layer).  The result is written
to gen/calibrated.py.  Run:  python -m gen.calibrate
"""
import os

import numpy as np

import gen

TARGET = {2: (2.0, 0.05), 4: (3.5, 0.1)}


def imbalance(cid, c_val):
    base = gen.WORKLOADS[cid]
    cfg = gen.Config(**{**base.__dict__, "bias_scale": c_val})
    return gen.rank_imbalance(cfg, gen.topk_all(cfg, 0))


def calibrate(cid, lo=0.0, hi=2.0, iters=30):
    target, tol = TARGET[cid]
    while imbalance(cid, hi) < target:
        hi *= 2
    for _ in range(iters):
        mid = 0.5 * (lo + hi)
        v = imbalance(cid, mid)
        if abs(v - target) <= tol / 4:
            return mid, v
        if v < target:
            lo = mid
        else:
            hi = mid
    mid = 0.5 * (lo + hi)
    return mid, imbalance(cid, mid)


def main():
    res = {}
    for cid in TARGET:
        c_val, v = calibrate(cid)
        print(f"config {cid}: c = {c_val!r} -> imbalance {v:.4f}")
        res[cid] = round(c_val, 6)
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "calibrated.py")
    with open(path, "w") as f:
        f.write('"""Frozen Zipf bias scales written by gen/calibrate.py."""\n')
        f.write(f"ZIPF_C = {res!r}\n")


if __name__ == "__main__":
    main()
