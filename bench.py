"""Benchmark of the Ball Sparse Attention layer hot path on one MI355X.

One step = ball-tree ordering of a 65536-point cloud, ordering of its Q/K/V rows and
gate logits, the layer forward pass and the layer backward pass (all on the GPU, all
through the C ABI). Inputs are seeded synthetic data already resident in HBM: a
32-component Gaussian mixture cloud, Q/K/V ~ N(0,1) in bf16, 8 heads of dim 64, ball
256, compression blocks of 16, selection blocks of 32, top-16, groups of 16.

Prints one JSON line (rank 0, N=1). Usage: python bench.py [--steps K] [--warmup W]
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

MFMA_BF16_PEAK = 2.5e15     # MI355X dense bf16 MFMA, FLOP/s
HBM_PEAK = 8.0e12           # MI355X HBM3E, B/s


def algorithmic_flops(cfg):
    """Work the method must do (not the dense work it avoids), per step.

    Per head: ball 4 N m d; MLP 2 (N/l)(l d d + d d) per tensor (K and V); compressed
    attention 4 N (N/l) d; scoring 2 (N/g)(N/l) d; selection 4 N k* l' d. Backward: 2.5x
    each attention term (5 vs 2 matrix products), 2x the MLP, nothing for scoring.
    """
    B, H, N, d = cfg.batch, cfg.heads, cfg.n_pad, cfg.head_dim
    m, l, ls, k, g = cfg.ball, cfg.cmp_block, cfg.slc_block, cfg.topk, cfg.group
    per = {
        "ball": 4.0 * N * m * d,
        "mlp": 2 * 2.0 * (N / l) * (l * d * d + d * d),
        "cmp": 4.0 * N * (N / l) * d,
        "score": 2.0 * (N / g) * (N / l) * d,
        "slc": 4.0 * N * k * ls * d,
    }
    fwd = {n: v * B * H for n, v in per.items()}
    bwd = {"ball": 2.5 * fwd["ball"], "mlp": 2 * fwd["mlp"], "cmp": 2.5 * fwd["cmp"], "score": 0.0,
           "slc": 2.5 * fwd["slc"]}
    return fwd, bwd


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", type=int, default=3)
    ap.add_argument("--cpu-baseline", type=int, default=1, help="time the float64 oracle on a sample (0 = skip)")
    return ap.parse_args()


def cpu_baseline(cfg, pts_np, inp_np):
    """The float64 oracle on a bounded sample of the same workload: the full ball tree
    plus one of the heads' forward and backward; the head time is scaled by the head
    count to give points/s for the whole step."""
    import numpy as np

    from oracle import bsa as ob
    from oracle.tree import build_ball_tree

    cores = len(os.sched_getaffinity(0))
    P = ob.Params(ball=cfg.ball, cmp_block=cfg.cmp_block, slc_block=cfg.slc_block, topk=cfg.topk, group=cfg.group)
    t0 = time.perf_counter()
    perm = build_ball_tree(pts_np[0], cfg.n_pad)
    t_tree = time.perf_counter() - t0
    h = 0
    sl = lambda a: np.ascontiguousarray(a[:, h:h + 1])
    valid = (perm >= 0)[None]
    q, k, v, do = (sl(inp_np[n]) for n in ("q", "k", "v", "do"))
    t0 = time.perf_counter()
    fwd = ob.forward(q, k, v, valid, inp_np["gate"], inp_np["phi_k"], inp_np["phi_v"], P)
    ob.backward(q, k, v, valid, inp_np["gate"], inp_np["phi_k"], inp_np["phi_v"], P, fwd, do)
    t_head = time.perf_counter() - t0
    total = t_tree + cfg.heads * t_head
    return {"value": cfg.batch * cfg.n_real / total, "unit": "points/s", "cores": cores, "kind": "oracle",
            "sample": f"ball tree of the full {cfg.n_real}-point cloud ({t_tree:.2f} s) + forward and backward of "
                      f"1 of {cfg.heads} heads ({t_head:.2f} s), scaled x{cfg.heads}; float64 numpy"}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for {args.gpus}); the multi-GPU sharding is a design "
              "in DESIGN.md, not a measured path", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2506_12541_amd import _lib
    from paper_2506_12541_amd import bsa as gb
    from workloads import CONFIGS, make_inputs, make_points

    cfg = CONFIGS[args.config]
    dev = torch.device("cuda:0")
    pts_np = make_points(cfg)
    inp_np = make_inputs(cfg, layout="points", with_grad=False)
    inp_np["do"] = make_inputs(cfg, layout="ball", with_grad=True)["do"]
    p = gb.Params.from_config(cfg)
    dt = p.torch_dtype
    t = lambda a, d=None: torch.from_numpy(np.ascontiguousarray(a)).to(dev).to(d or torch.float32)
    pts = t(pts_np)
    xq, xk, xv = (t(inp_np[n], dt) for n in ("q", "k", "v"))
    gate_pts = t(inp_np["gate"])
    phi_k = {w: t(a) for w, a in inp_np["phi_k"].items()}
    phi_v = {w: t(a) for w, a in inp_np["phi_v"].items()}
    dout = t(inp_np["do"], dt)
    saved = gb.Saved(p, dev)
    H, d = cfg.heads, cfg.head_dim

    def step():
        perm = gb.build_ball_tree(pts, cfg.n_pad)
        q, valid = gb.permute(xq, perm, H, d, with_valid=True)
        k = gb.permute(xk, perm, H, d)
        v = gb.permute(xv, perm, H, d)
        gate = gb.permute(gate_pts, perm, 1, 3).view(cfg.batch, cfg.n_pad, 3)
        # every slot holds a real point when n_real == n_pad: the layer may skip key masks
        vmask = None if cfg.n_real == cfg.n_pad else valid
        o, sv = gb.forward(p, q, k, v, vmask, gate, phi_k, phi_v, saved=saved)
        grads = gb.backward(p, q, k, v, vmask, gate, phi_k, phi_v, sv, dout)
        return o, grads

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    lib = _lib.load()
    lib.bsa_timing_enable(1)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    phases = {}
    for name in ("tree", "permute", "fwd.compress", "fwd.select", "fwd.ball", "fwd.cmp", "fwd.slc", "fwd.gate",
                 "bwd.gate", "bwd.dq_ball", "bwd.dq_cmp", "bwd.dq_slc", "bwd.kv_ball", "bwd.kv_cmp", "bwd.mlp",
                 "bwd.slc_csr", "bwd.slc_kv"):
        tot = _lib.C.c_double()
        cnt = _lib.C.c_int32()
        _lib.check(lib.bsa_timing_query(name.encode(), _lib.C.byref(tot), _lib.C.byref(cnt)), "timing")
        phases[name] = tot.value / max(1, args.steps)
    lib.bsa_timing_enable(0)

    ms = elapsed / args.steps * 1e3
    fwd_f, bwd_f = algorithmic_flops(cfg)
    flops = sum(fwd_f.values()) + sum(bwd_f.values())
    layer_ms = sum(v for n, v in phases.items() if n.startswith(("fwd.", "bwd.")))
    tflops = flops / (layer_ms * 1e-3) / 1e12
    # dominant kernel: the compressed-attention forward kernel (4 N (N/l) d per head)
    cmp_ms = phases["fwd.cmp"]
    cmp_flops = fwd_f["cmp"]
    achieved = cmp_flops / (cmp_ms * 1e-3) / 1e12
    result = {
        "metric": "BSA layer fwd+bwd points/sec and TFLOP/s (fraction of MFMA peak) at N=65536, 1 GPU",
        "value": cfg.batch * cfg.n_real / (ms * 1e-3),
        "unit": "points/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"{cfg.name}: {cfg.batch}x{cfg.n_real} points (32-component Gaussian mixture), "
                               f"H={cfg.heads} d={cfg.head_dim}, ball {cfg.ball}, cmp block {cfg.cmp_block}, "
                               f"slc block {cfg.slc_block}, top-{cfg.topk}, group {cfg.group}; tree + permute + "
                               f"forward + backward",
                   "points": cfg.batch * cfg.n_real, "heads": cfg.heads, "head_dim": cfg.head_dim},
        "tflops": tflops,
        "mfma_frac": tflops * 1e12 / MFMA_BF16_PEAK,
        "algorithmic_gflop_per_step": flops / 1e9,
        "phase_ms": {n: round(v, 4) for n, v in phases.items()},
        "roofline": {"bound": "mfma", "kernel": "compressed-attention forward (fwd.cmp)", "achieved": achieved,
                     "peak": MFMA_BF16_PEAK / 1e12, "unit": "TFLOP/s", "frac": achieved * 1e12 / MFMA_BF16_PEAK,
                     "traffic": None},
    }
    if args.cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(cfg, pts_np, {**inp_np, **make_inputs(cfg, layout="ball",
                                                                                     with_grad=True)})
    print(json.dumps(result))


if __name__ == "__main__":
    main()
