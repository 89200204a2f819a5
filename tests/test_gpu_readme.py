"""The usage example of README.md, executed as written on a small workload
(the buffers it names are supplied here), its results compared with the
oracle.  Needs an MI355X."""
import os
import re

import numpy as np
import pytest
import torch

import gen
import oracle

pytestmark = pytest.mark.gpu

README = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "README.md")


def _example():
    text = open(README).read()
    sec = text[text.index("## Using the library"):]
    return re.search(r"```python\n(.*?)```", sec, re.S).group(1)


def test_readme_example_runs_and_matches_the_oracle():
    c = gen.config(2)
    R, E, n_slot, u_min, T, k, H = c.R, c.E, c.n_slot, c.u_min, c.T, c.k, c.H
    W = 8 * 1024
    dev = torch.device("cuda")
    tk_all = gen.topk_all(c, 0)
    og = oracle.Group(R, E, n_slot, u_min, 101, 100)
    oload, _ = oracle.count(tk_all, E, R)
    op = oracle.plan(oload, og)
    X = op.slot_expert
    rank = int(np.argmax([((X >= 0) & (X // c.n_main == r)).sum() for r in range(R)]))
    x_h = gen.activations(c, 0, rank)
    w_h = gen.weights(c, rank, W=W)
    rng = np.random.default_rng(5)
    gate_h = rng.random((T, k)).astype(np.float32)
    y_h = rng.integers(0, 1 << 16, (T * k, H)).astype(np.uint16)
    cap = R * n_slot
    load = torch.from_numpy(oload.copy()).to(dev)
    load[rank] = -1  # the example recounts this rank's row
    ns = dict(R=R, E=E, n_slot=n_slot, u_min=u_min, T=T, k=k, H=H, W=W, rank=rank, cap=cap,
              topk=torch.from_numpy(tk_all[rank].copy()).to(dev), load=load,
              w_main=torch.from_numpy(w_h.view(np.int16)).to(dev),
              staging=torch.zeros((cap, W), dtype=torch.int16, device=dev),
              dest_off=torch.empty(R + 1, dtype=torch.int64, device=dev),
              row_of_slot=torch.empty(T * k, dtype=torch.int32, device=dev),
              block_off=torch.empty(R * (E // R + n_slot) + 1, dtype=torch.int64, device=dev),
              x=torch.from_numpy(x_h.view(np.int16)).to(dev),
              send=torch.empty((T * k, H), dtype=torch.int16, device=dev),
              y=torch.from_numpy(y_h.view(np.int16)).to(dev),
              gate=torch.from_numpy(gate_h).to(dev),
              out=torch.empty((T, H), dtype=torch.int16, device=dev))
    exec(compile(_example(), "README.md", "exec"), ns)
    assert np.array_equal(ns["load"].cpu().numpy(), oload)
    osend, oros, oboff, st = oracle.dispatch(x_h, tk_all[rank], rank, og, op)
    assert st == 0
    assert np.array_equal(ns["row_of_slot"].cpu().numpy(), oros)
    assert np.array_equal(ns["block_off"].cpu().numpy(), oboff)
    assert np.array_equal(ns["send"].cpu().numpy().view(np.uint16), osend)
    ostg, odoff, n_out, st = oracle.pack(w_h, rank, og, op, cap)
    assert st == 0
    assert np.array_equal(ns["dest_off"].cpu().numpy(), odoff)
    assert np.array_equal(ns["staging"][:n_out].cpu().numpy().view(np.uint16), ostg[:n_out])
    oout, st = oracle.combine(y_h, gate_h, oros)
    assert st == 0
    assert np.array_equal(ns["out"].cpu().numpy().view(np.uint16), oout)
