"""Shared helpers of the GPU parity tests: run the HIP path through the C ABI, run the
float64 oracle on the same seeded inputs, and compare with the stated tolerances."""
from __future__ import annotations

import numpy as np
import torch

from oracle import bsa as ob
from oracle.tree import build_ball_tree
from paper_2506_12541_amd import bsa as gb
from workloads import make_inputs, make_points

TOL = {"f32": 1e-4, "bf16": 2e-2}   # max-abs output tolerance per storage type
TIE = 1e-6                          # score gap under which two blocks count as tied


# C-side variant parameters -> oracle Params keywords
def oracle_kw(pkw) -> dict:
    okw = {}
    if pkw.get("kv_pool") == 1:
        okw["kv_pool"] = "mean"
    if pkw.get("mask_own_ball") == 0:
        okw["mask_own_ball"] = False
    if pkw.get("q_coarsen") == 1:
        okw["q_coarsen"] = "mlp"
    if pkw.get("group_compression") == 1:
        okw["group_compression"] = True
    return okw


def oracle_params(cfg, **kw) -> ob.Params:
    return ob.Params(ball=cfg.ball, cmp_block=cfg.cmp_block, slc_block=cfg.slc_block, topk=cfg.topk,
                     group=cfg.group, **kw)


def valid_from_tree(cfg, seed=None) -> np.ndarray:
    """Real/padding slots of each cloud, from the oracle's tree on the config's points."""
    if cfg.n_real == cfg.n_pad:
        return np.ones((cfg.batch, cfg.n_pad), bool)
    pts = make_points(cfg, seed)
    return np.stack([build_ball_tree(pts[b], cfg.n_pad) >= 0 for b in range(cfg.batch)])


def to_dev(x, dtype):
    return torch.from_numpy(np.ascontiguousarray(x)).to("cuda").to(dtype)


def gpu_forward(cfg, inp, valid, **pkw):
    p = gb.Params.from_config(cfg, **pkw)
    dt = p.torch_dtype
    q, k, v = (to_dev(inp[n], dt) for n in ("q", "k", "v"))
    gate = to_dev(inp["gate"], torch.float32)
    # every slot real: no mask, as the benchmark launches the layer (the unmasked kernels)
    vd = None if valid is None or valid.all() else to_dev(valid.astype(np.uint8), torch.uint8)
    phi_k = {w: to_dev(a, torch.float32) for w, a in inp["phi_k"].items()}
    phi_v = {w: to_dev(a, torch.float32) for w, a in inp["phi_v"].items()}
    phi_q = {w: to_dev(a, torch.float32) for w, a in inp["phi_q"].items()}
    o, saved = gb.forward(p, q, k, v, vd, gate, phi_k, phi_v, phi_q=phi_q)
    torch.cuda.synchronize()
    f = lambda t: t.float().cpu().numpy()
    lse = saved.lse.cpu().numpy() if saved.lse is not None else None
    return {"o": f(o), "o_branch": f(saved.branch_outputs()), "lse": lse,
            "sel": saved.sel_idx.cpu().numpy().astype(np.int64), "kc": saved.kcmp.cpu().numpy(),
            "vc": saved.vcmp.cpu().numpy(), "qc": saved.qcmp.cpu().numpy()}, \
        (p, q, k, v, vd, gate, phi_k, phi_v, saved, o, phi_q)


def check_indices(sel_gpu, sel_or, scores):
    """Bit-exact selected blocks, except where every differing block is within TIE of the
    oracle's k-th score. Returns the number of rows that differ (all of them tie-justified)."""
    assert sel_gpu.shape == sel_or.shape
    k = sel_or.shape[-1]
    diff_rows = 0
    flat_g = sel_gpu.reshape(-1, k)
    flat_o = sel_or.reshape(-1, k)
    flat_s = scores.reshape(-1, scores.shape[-1])
    for r in np.nonzero(np.any(flat_g != flat_o, axis=1))[0]:
        g = set(int(x) for x in flat_g[r] if x >= 0)
        o = set(int(x) for x in flat_o[r] if x >= 0)
        assert len(g) == len(o), (r, flat_g[r], flat_o[r])
        assert list(flat_g[r]) == sorted(g) + [-1] * (k - len(g)), "GPU row not ascending/-1 padded"
        kth = np.sort(flat_s[r][np.isfinite(flat_s[r])])[::-1][len(o) - 1]
        for blk in g ^ o:
            assert abs(flat_s[r][blk] - kth) < TIE, (r, blk, flat_s[r][blk], kth)
        diff_rows += 1
    return diff_rows


def max_abs(a, b, mask=None):
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    with np.errstate(invalid="ignore"):
        d = np.where(a == b, 0.0, np.abs(a - b))   # equal infinities (no key: lse -inf) agree
    if mask is not None:
        d = d[mask]
    return float(d.max()) if d.size else 0.0
