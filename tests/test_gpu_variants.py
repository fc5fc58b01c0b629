"""GPU vs float64 oracle for the layer variants of Section 2.2: query coarsening by an MLP
phi_q over blocks of l queries (Eq. 13-14) and group compression (Eq. 15), forward and
backward, on the same seeded inputs.

Bars as for the regular layer: coarse queries within 1e-4 of the oracle's (they are
float32 on the GPU); selected blocks bit-exact except where the oracle's own scores tie
within 1e-6; branch outputs (with the GPU's selection), LSE and the gated output at
max-abs 1e-4 (f32) / 2e-2 (bf16); dQ, dK, dV at the same max-abs; gate-logit and MLP
weight gradients relative to the magnitude of their summed terms."""
import dataclasses

import numpy as np
import pytest

from oracle import bsa as ob
from parity import TOL, check_indices, gpu_forward, max_abs, oracle_kw, oracle_params, valid_from_tree
from test_gpu_backward import run_case
from workloads import CONFIGS, Config, make_inputs

pytestmark = pytest.mark.gpu

VARIANTS = [dict(q_coarsen=1, group_compression=1), dict(group_compression=1), dict(q_coarsen=1)]
IDS = ["mlp_coarsen+group_cmp", "mean+group_cmp", "mlp_coarsen"]

# 2 clouds of 900 points in 1024 slots, d = 64, l = g = 16: 64 coarse queries per head
# (the smallest group-compression grid: one 64-row tile), ragged padding
SMALL = Config("small_bf16", 2, 900, 1024, 2, 64, "bf16", 128, 16, 16, 32, 4, 16, "uniform", "fwdbwd")


def _f64(x):
    return np.asarray(x, np.float64)


def _check_head(inp, valid, g, b, h, P, tol, groups=None):
    q, k, v = (_f64(inp[n][b, h]) for n in ("q", "k", "v"))
    phk, phv, phq = ({w: _f64(a) for w, a in inp[n].items()} for n in ("phi_k", "phi_v", "phi_q"))
    vb = valid[b]
    n, d = q.shape
    kc, _ = ob.compress(k, vb, phk, P)
    vc, _ = ob.compress(v, vb, phv, P)
    qc, _ = ob.coarse_queries(q, vb, phq, P)
    assert max_abs(g["kc"][b, h], kc) < 1e-4 and max_abs(g["vc"][b, h], vc) < 1e-4
    assert max_abs(g["qc"][b, h], qc) < 1e-4
    gsel = g["sel"][b, h]
    if groups is None:
        groups = np.arange(n // P.group)
    rows = (groups[:, None] * P.group + np.arange(P.group)[None, :]).reshape(-1)
    scores = ob.group_block_scores(q, kc, vb, P, groups=groups, qc=qc)
    ndiff = check_indices(gsel[groups], ob.topk_blocks(scores, P.topk), scores)
    rv = np.zeros(n, bool)
    rv[rows] = True
    rv &= vb
    o_ball, l_ball = np.zeros((n, d)), np.full(n, -np.inf)
    for s0 in np.unique((rows // P.ball) * P.ball):
        sl = slice(s0, s0 + P.ball)
        o_ball[sl], l_ball[sl] = ob.ball_branch(q[sl], k[sl], v[sl], vb[sl], P)
    cvalid = ob.block_valid(vb, P.cmp_block)
    if P.group_compression:
        o_cmp, l_cmp, _, _ = ob.group_compression_branch(qc, kc, vc, cvalid, vb, P)
    else:
        o_cmp, l_cmp = ob.compression_branch(q, kc, vc, cvalid, vb, P, rows=rows)
    o_slc, l_slc = ob.selection_branch(q, k, v, vb, gsel, P, groups=groups)
    outs, lses = (o_ball, o_cmp, o_slc), (l_ball, l_cmp, l_slc)
    for br in range(3):
        err = max_abs(g["o_branch"][br, b, h], outs[br], rv)
        assert err < tol, (br, err)
        assert max_abs(g["lse"][br, b, h], lses[br], rv) < tol, br
        assert not np.any(g["o_branch"][br, b, h][~vb]), "padding rows must be zero"
    sg = 1.0 / (1.0 + np.exp(-_f64(inp["gate"][b])))
    o = sum(sg[:, br, None] * outs[br] for br in range(3))
    assert max_abs(g["o"][b, h], o, rv) < tol
    return ndiff


@pytest.mark.parametrize("pkw", VARIANTS, ids=IDS)
@pytest.mark.parametrize("cfg_id", [1, 2])
def test_variant_forward(cfg_id, pkw):
    cfg = CONFIGS[cfg_id]
    print(f"variant forward parity config {cfg_id} {pkw}", flush=True)
    inp = make_inputs(cfg, layout="ball", with_grad=False)
    valid = valid_from_tree(cfg)
    if cfg.n_real == cfg.n_pad:      # add padding slots (incl. one whole empty block)
        valid = valid.copy()
        valid[0, 100:140] = False
    g, _ = gpu_forward(cfg, inp, valid, **pkw)
    P = oracle_params(cfg, **oracle_kw(pkw))
    ndiff = 0
    for b in range(min(cfg.batch, 4)):
        for h in range(cfg.heads):
            ndiff += _check_head(inp, valid, g, b, h, P, TOL[cfg.dtype])
    print(f"tie-justified index differences: {ndiff} rows")


@pytest.mark.parametrize("pkw", VARIANTS[:2], ids=IDS[:2])
def test_variant_forward_small_tile(pkw):
    print(f"variant forward parity small bf16 d=64 {pkw}", flush=True)
    inp = make_inputs(SMALL, seed=11, layout="ball", with_grad=False)
    valid = valid_from_tree(SMALL, seed=11)
    g, _ = gpu_forward(SMALL, inp, valid, **pkw)
    P = oracle_params(SMALL, **oracle_kw(pkw))
    for b in range(SMALL.batch):
        for h in range(SMALL.heads):
            _check_head(inp, valid, g, b, h, P, TOL["bf16"])


@pytest.mark.timeout(300)
def test_group_compression_scaling_sampled():
    """The 65536-point workload with MLP coarsening and group compression; oracle on 64
    sampled groups of two heads (coarse attention of every block of those heads)."""
    cfg = CONFIGS[3]
    pkw = dict(q_coarsen=1, group_compression=1)
    print("variant forward parity config 3 (sampled)", flush=True)
    inp = make_inputs(cfg, layout="ball", with_grad=False)
    valid = valid_from_tree(cfg)
    g, _ = gpu_forward(cfg, inp, valid, **pkw)
    P = oracle_params(cfg, **oracle_kw(pkw))
    rng = np.random.default_rng(5)
    ngroups = cfg.n_pad // cfg.group
    for h in (1, cfg.heads - 2):
        groups = np.unique(np.concatenate([[0, ngroups - 1], rng.choice(ngroups, 62, replace=False)]))
        _check_head(inp, valid, g, 0, h, P, TOL[cfg.dtype], groups=groups)


@pytest.mark.parametrize("pkw", VARIANTS[:2], ids=IDS[:2])
def test_variant_backward_fp32(pkw):
    print(f"variant backward parity config 1 {pkw}", flush=True)
    run_case(CONFIGS[1], **pkw)


@pytest.mark.parametrize("pkw", VARIANTS[:2], ids=IDS[:2])
def test_variant_backward_airflow_bf16(pkw):
    print(f"variant backward parity config 5 {pkw}", flush=True)
    run_case(CONFIGS[5], **pkw)


def test_variant_backward_small_tile():
    print("variant backward parity small bf16 d=64, mlp coarsening + group compression", flush=True)
    run_case(SMALL, seed=11, q_coarsen=1, group_compression=1)


def test_mlp_coarsening_backward_leaves_phi_q():
    # without group compression phi_q only feeds the (gradient-free) top-k: the layer's
    # gradients are those of the regular layer with the same selection
    print("variant backward parity config 1, mlp coarsening only", flush=True)
    run_case(CONFIGS[1], q_coarsen=1)


# ---- per-token selection (g = 1: Eq. 6-8 without the grouping of Eq. 10-12) ----

@pytest.mark.parametrize("cfg", [dataclasses.replace(CONFIGS[2], group=1, batch=4),
                                 dataclasses.replace(SMALL, group=1)], ids=["airflow_l16", "small_l32"])
def test_per_token_forward(cfg):
    print(f"per-token selection forward parity {cfg.name} group 1", flush=True)
    inp = make_inputs(cfg, seed=7, layout="ball", with_grad=False)
    valid = valid_from_tree(cfg, seed=7)
    g, _ = gpu_forward(cfg, inp, valid)
    P = oracle_params(cfg)
    ndiff = 0
    for b in range(min(cfg.batch, 2)):
        for h in range(cfg.heads):
            ndiff += _check_head(inp, valid, g, b, h, P, TOL[cfg.dtype])
    print(f"tie-justified index differences: {ndiff} rows")


@pytest.mark.timeout(300)
def test_per_token_scaling_sampled():
    """The 65536-point workload with per-token selection; oracle on 256 sampled queries of
    two heads."""
    cfg = dataclasses.replace(CONFIGS[3], group=1)
    print("per-token selection forward parity 65536 points (sampled)", flush=True)
    inp = make_inputs(cfg, seed=3, layout="ball", with_grad=False)
    valid = valid_from_tree(cfg, seed=3)
    g, _ = gpu_forward(cfg, inp, valid)
    P = oracle_params(cfg)
    rng = np.random.default_rng(6)
    for h in (0, cfg.heads - 1):
        groups = np.unique(np.concatenate([[0, cfg.n_pad - 1], rng.choice(cfg.n_pad, 254, replace=False)]))
        _check_head(inp, valid, g, 0, h, P, TOL[cfg.dtype], groups=groups)


@pytest.mark.parametrize("cfg", [dataclasses.replace(CONFIGS[5], group=1, batch=2),
                                 dataclasses.replace(SMALL, group=1)], ids=["airflow_l16", "small_l32"])
def test_per_token_backward(cfg):
    print(f"per-token selection backward parity {cfg.name} group 1", flush=True)
    run_case(cfg, seed=9)
