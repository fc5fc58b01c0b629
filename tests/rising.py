"""Inputs whose attention scores rise along the key order, for the forward parity test of
the online softmax's moving reference maximum. Input construction only: no GPU code and
none of the layer's arithmetic."""
import dataclasses

import numpy as np

from workloads import CONFIGS, make_inputs, round_bf16


def rising_config(dtype="bf16"):
    """An unmasked layer of 8192 points and two heads, shaped like the 65536-point
    workload otherwise (ball 256, compression blocks of 16, selection blocks of 32); head
    dim 64 for bf16 layers, 32 for float32 ones (the float32 kernels' only head dim)."""
    return dataclasses.replace(CONFIGS[3], name=f"rising_8192_{dtype}", n_real=8192, n_pad=8192, heads=2,
                               head_dim=64 if dtype == "bf16" else 32, dtype=dtype, passes="fwd")


def rising_inputs(cfg):
    """The seeded inputs of `cfg` with queries 1 + 0.05 x and keys c(t) + 0.05 x, where
    c(t) = (8/sqrt(d)) (3 ((t mod m)/m - 1/2) + 6 (t/N - 1/2)) rises inside each ball and
    along the cloud, by the same scores at every head dim d
    (x: the seeded N(0,1) draws); bf16-representable for bf16 layers, as their other
    inputs."""
    inp = make_inputs(cfg, layout="ball", with_grad=False)
    n = cfg.n_pad
    t = np.arange(n)
    c = 8.0 / np.sqrt(cfg.head_dim) * (3.0 * ((t % cfg.ball) / cfg.ball - 0.5) + 6.0 * (t / n - 0.5))
    rnd = round_bf16 if cfg.dtype == "bf16" else (lambda a: a)
    inp["k"] = rnd((c[None, None, :, None] + 0.05 * inp["k"]).astype(np.float32))
    inp["q"] = rnd((1.0 + 0.05 * inp["q"]).astype(np.float32))
    return inp
