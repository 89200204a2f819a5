"""Seeded synthetic workloads shaped like the paper's MoE layers.

This module is the one input source shared by the tests and the benchmark.  It
holds none of the balancing method's arithmetic: it draws router logits, picks
top-k experts per token, and fills activations and expert weights.

The paper's own routing traces, corpora and serving datasets are not
available; the router below stands in for them with the shapes of the
evaluated models (experts, top-k, EP size, redundant slots) and with the load
phenomena the paper reports: power-law skew, drift across microbatches and
hot-expert bursts (Sec. 3, Sec. 8.5).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass, field

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "gen.c")
_LIB = os.path.join(_HERE, "libultraep_gen.so")

# stream labels
S_LOGITS, S_BIAS, S_ACT, S_WEIGHT, S_BURST = 0, 1, 2, 3, 4


def build() -> str:
    cmd = ["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared", "-o",
           _LIB + ".tmp", _SRC, "-lm"]
    subprocess.run(cmd, check=True, cwd=_HERE)
    os.replace(_LIB + ".tmp", _LIB)
    return _LIB


_lib = None
_P = ctypes.c_void_p


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        L = ctypes.CDLL(_LIB)
        u64, i64, i32 = ctypes.c_uint64, ctypes.c_int64, ctypes.c_int32
        L.gen_key.argtypes = [u64] * 5
        L.gen_key.restype = u64
        L.gen_normals.argtypes = [u64, i64, _P]
        L.gen_bf16_normals.argtypes = [u64, i64, _P]
        L.gen_bits16.argtypes = [u64, i64, _P]
        L.gen_perm.argtypes = [u64, i32, _P]
        L.gen_router_topk.argtypes = [u64, i64, i64, i32, i32, _P, i32, i32, _P]
        L.gen_router_topk.restype = ctypes.c_int
        _lib = L
    return _lib


def key(seed, a=0, b=0, c=0, d=0) -> int:
    return lib().gen_key(seed, a, b, c, d)


def normals(k, n):
    out = np.empty(n, np.float64)
    lib().gen_normals(k, n, out.ctypes.data_as(_P))
    return out


def bf16_normals(k, shape):
    out = np.empty(shape, np.uint16)
    lib().gen_bf16_normals(k, out.size, out.ctypes.data_as(_P))
    return out


def bits16(k, shape):
    out = np.empty(shape, np.uint16)
    lib().gen_bits16(k, out.size, out.ctypes.data_as(_P))
    return out


def perm(k, n):
    out = np.empty(n, np.int32)
    lib().gen_perm(k, n, out.ctypes.data_as(_P))
    return out


def router_topk(k_logits, tok0, n_tok, E, k, bias, n_group=0, top_group=0):
    bias = np.ascontiguousarray(bias, np.float64)
    assert bias.shape == (E,)
    out = np.empty((n_tok, k), np.int32)
    rc = lib().gen_router_topk(k_logits, tok0, n_tok, E, k,
                               bias.ctypes.data_as(_P), n_group, top_group,
                               out.ctypes.data_as(_P))
    assert rc == 0, "bad router arguments"
    return out


@dataclass(frozen=True)
class Config:
    """One synthetic workload: EP group shape, router model and tensor sizes."""
    cid: int
    name: str
    R: int
    E: int
    n_slot: int
    k: int
    T: int          # tokens per rank per microbatch
    H: int          # hidden size (bf16 row = 2*H bytes)
    F: int          # expert FFN width; an expert blob is 3*H*F bf16
    u_min: int
    bias: str       # "normal" | "zipf" | "drift" | "burst"
    bias_scale: float = 0.0   # normal: sigma; zipf: calibrated c; drift: step
    zipf_s: float = 0.0
    n_group: int = 0
    top_group: int = 0
    n_micro: int = 1          # microbatches (drift) or layers (burst)
    burst_n: int = 0
    burst_b: float = 0.0
    beta_num: int = 101
    beta_den: int = 100

    @property
    def seed(self) -> int:
        return 4101 + self.cid

    @property
    def n_main(self) -> int:
        return self.E // self.R

    @property
    def W(self) -> int:
        """bf16 elements per expert blob (gate H x F, up H x F, down F x H)."""
        return 3 * self.H * self.F


# The five workloads.  Expert counts, top-k, EP sizes and redundant slots
# follow Table 2 / Sec. 8.1 of the paper; the Zipf scales c are calibrated
# once (gen/calibrate.py) so that microbatch 0 has the stated max/mean rank
# load, then frozen here.
WORKLOADS = {
    1: Config(1, "tiny", R=4, E=16, n_slot=2, k=2, T=512, H=256, F=512,
              u_min=32, bias="normal", bias_scale=1.5),
    2: Config(2, "glm45air_layer", R=32, E=128, n_slot=2, k=8, T=4096,
              H=4096, F=1408, u_min=1024, bias="zipf", zipf_s=1.1,
              bias_scale=0.0),
    3: Config(3, "qwen3_235b_layer", R=64, E=128, n_slot=2, k=8, T=8192,
              H=4096, F=1536, u_min=1024, bias="drift", bias_scale=0.3,
              n_micro=16),
    4: Config(4, "dsv3_train_layer", R=64, E=256, n_slot=1, k=8, T=4096,
              H=7168, F=2048, u_min=1024, bias="zipf", zipf_s=1.3,
              bias_scale=0.0, n_group=8, top_group=4),
    5: Config(5, "dsv3_prefill_layers", R=32, E=256, n_slot=2, k=8, T=16384,
              H=7168, F=2048, u_min=1024, bias="burst", n_group=8,
              top_group=4, n_micro=58, burst_n=8, burst_b=3.0),
}

# calibrated Zipf scales (see gen/calibrate.py); filled in below
ZIPF_C = {2: None, 4: None}


def config(cid: int) -> Config:
    c = WORKLOADS[cid]
    if c.bias == "zipf":
        cc = ZIPF_C[cid]
        if cc is None:
            raise RuntimeError(f"config {cid}: Zipf scale not calibrated")
        c = Config(**{**c.__dict__, "bias_scale": cc})
    return c


def bias(c: Config, m: int = 0) -> np.ndarray:
    """Per-expert router bias for microbatch (or layer) m."""
    E = c.E
    if c.bias == "normal":
        return c.bias_scale * normals(key(c.seed, S_BIAS), E)
    if c.bias == "zipf":
        rho = perm(key(c.seed, S_BIAS), E).astype(np.float64) + 1.0
        return -c.bias_scale * c.zipf_s * np.log(rho)
    if c.bias == "drift":
        b = normals(key(c.seed, S_BIAS, 0), E)
        for i in range(1, m + 1):
            b = b + c.bias_scale * normals(key(c.seed, S_BIAS, i), E)
        return b
    if c.bias == "burst":
        p = perm(key(c.seed, S_BURST, m), E)[: c.burst_n]
        b = np.zeros(E)
        b[p] = c.burst_b
        return b
    raise ValueError(c.bias)


def topk_rank(c: Config, m: int, r: int, b=None) -> np.ndarray:
    """[T, k] int32 expert ids of rank r's tokens in microbatch/layer m."""
    if b is None:
        b = bias(c, m)
    kl = key(c.seed, S_LOGITS, m)
    return router_topk(kl, r * c.T, c.T, c.E, c.k, b, c.n_group, c.top_group)


def topk_all(c: Config, m: int = 0) -> np.ndarray:
    """[R, T, k] int32: every simulated rank's routing for microbatch m."""
    b = bias(c, m)
    kl = key(c.seed, S_LOGITS, m)
    out = router_topk(kl, 0, c.R * c.T, c.E, c.k, b, c.n_group, c.top_group)
    return out.reshape(c.R, c.T, c.k)


def activations(c: Config, m: int, r: int, T: int | None = None) -> np.ndarray:
    """[T, H] bf16 (as uint16) N(0,1) token rows of rank r."""
    return bf16_normals(key(c.seed, S_ACT, m, r), (T or c.T, c.H))


def weights(c: Config, r: int, n_main: int | None = None, W: int | None = None):
    """[n_main, W] uint16: rank r's main-expert blobs as raw bit patterns."""
    return bits16(key(c.seed, S_WEIGHT, r), (n_main or c.n_main, W or c.W))


def rank_imbalance(c: Config, topk_all_ranks: np.ndarray) -> float:
    """max/mean rank load of a routing (workload statistic for calibration)."""
    ids = topk_all_ranks.reshape(-1)
    per_expert = np.bincount(ids[ids >= 0], minlength=c.E)
    per_rank = per_expert.reshape(c.R, c.n_main).sum(1)
    return float(per_rank.max() / per_rank.mean())


from .calibrated import ZIPF_C as _ZC  # noqa: E402

ZIPF_C.update(_ZC)
