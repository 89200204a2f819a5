"""bench.py's parts that need no GPU: more than one GPU is refused with a
message and exit status 2, before any device work; the algorithmic bytes its
roofline divides by."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    for n in (2, 8):
        r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", str(n)],
                           capture_output=True, text=True, timeout=300)
        assert r.returncode == 2
        assert "one GPU only" in r.stderr
        assert r.stdout == ""


def test_algorithmic_bytes_of_the_bench_layer():
    """The bytes the roofline divides by, on the DeepSeek-V3-shaped training
    layer and its rank with the most outbound replicas (the oracle's plan):
    the scatter moves 2·T·H + 2·n_routed·H + 4·T·k = 58.7 + 469.8 + 0.13 MB
    and the packing ships one expert blob of W_e = 3·H·F·2 bytes twice, so it
    reads W_e once and writes it twice."""
    import numpy as np
    sys.path.insert(0, ROOT)
    import bench
    import gen
    import oracle
    c = gen.config(4)
    tk = gen.topk_all(c, 0)
    load, st = oracle.count(tk, c.E, c.R)
    assert st == 0
    op = oracle.plan(load, oracle.Group(c.R, c.E, c.n_slot, c.u_min, c.beta_num, c.beta_den))
    X = op.slot_expert.reshape(c.R, c.n_slot)
    rank = int(np.argmax([((X >= 0) & (X // c.n_main == r)).sum() for r in range(c.R)]))
    fan = bench.outbound_fan(X, c.n_main, rank)
    assert sorted(int(f) for f in fan if f) == [2]
    n_routed = int((tk[rank] >= 0).sum())
    assert n_routed == c.T * c.k
    W_e = 3 * c.H * c.F * 2
    assert c.W * 2 == W_e == 88_080_384
    scatter, pack = bench.algorithmic_bytes(c.T, c.H, c.k, n_routed, c.W, fan)
    assert scatter == 528_613_376
    assert pack == 3 * W_e == 264_241_152
