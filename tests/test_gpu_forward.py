"""GPU forward pass vs the float64 oracle on the same seeded inputs.

Selected blocks must match bit-exactly except where the oracle's own scores tie within
1e-6; branch outputs are compared with the oracle re-run on the GPU's selection, at
max-abs 1e-4 (f32 layers) or 2e-2 (bf16 layers)."""
import dataclasses

import numpy as np
import pytest

from oracle import bsa as ob
from parity import TOL, check_indices, gpu_forward, max_abs, oracle_params, valid_from_tree
from rising import rising_config, rising_inputs
from workloads import CONFIGS, make_inputs

pytestmark = pytest.mark.gpu


def _f64(x):
    return np.asarray(x, np.float64)


def _check_head(cfg, inp, valid, g, b, h, P, tol, groups=None):
    q, k, v = (_f64(inp[n][b, h]) for n in ("q", "k", "v"))
    phk = {w: _f64(a) for w, a in inp["phi_k"].items()}
    phv = {w: _f64(a) for w, a in inp["phi_v"].items()}
    vb = valid[b]
    kc, _ = ob.compress(k, vb, phk, P)
    vc, _ = ob.compress(v, vb, phv, P)
    assert max_abs(g["kc"][b, h], kc) < 1e-4 and max_abs(g["vc"][b, h], vc) < 1e-4
    n = q.shape[0]
    gsel = g["sel"][b, h]
    if groups is None:
        groups = np.arange(n // P.group)
        rows = np.arange(n)
    else:
        rows = (groups[:, None] * P.group + np.arange(P.group)[None, :]).reshape(-1)
    scores = ob.group_block_scores(q, kc, vb, P, groups=groups)
    osel = ob.topk_blocks(scores, P.topk)
    ndiff = check_indices(gsel[groups], osel, scores)
    # branch outputs given the GPU's selection
    rmask = np.zeros(n, bool)
    rmask[rows] = True
    rv = rmask & vb
    if rows.size < n:     # sampled rows: ball attention only for the balls they touch
        o_ball, l_ball = np.zeros((n, q.shape[1])), np.full(n, -np.inf)
        for s0 in np.unique((rows // P.ball) * P.ball):
            sl = slice(s0, s0 + P.ball)
            o_ball[sl], l_ball[sl] = ob.ball_branch(q[sl], k[sl], v[sl], vb[sl], P)
    else:
        o_ball, l_ball = ob.ball_branch(q, k, v, vb, P)
    o_cmp, l_cmp = ob.compression_branch(q, kc, vc, ob.block_valid(vb, P.cmp_block), vb, P, rows=rows)
    o_slc, l_slc = ob.selection_branch(q, k, v, vb, gsel, P, groups=groups)
    outs = (o_ball, o_cmp, o_slc)
    lses = (l_ball, l_cmp, l_slc)
    for br in range(3):
        err = max_abs(g["o_branch"][br, b, h], outs[br], rv)
        assert err < tol, (br, err)
        assert max_abs(g["lse"][br, b, h], lses[br], rv) < tol, br
        assert not np.any(g["o_branch"][br, b, h][rmask & ~vb]), "padding rows must be zero"
    sg = 1.0 / (1.0 + np.exp(-_f64(inp["gate"][b])))
    o = sum(sg[:, br, None] * outs[br] for br in range(3))
    assert max_abs(g["o"][b, h], o, rv) < tol
    assert not np.any(g["o"][b, h][rmask & ~vb])
    return ndiff


@pytest.mark.parametrize("cfg_id", [1, 2])
def test_forward_full(cfg_id):
    cfg = CONFIGS[cfg_id]
    print(f"forward parity config {cfg_id}", flush=True)
    inp = make_inputs(cfg, layout="ball", with_grad=False)
    valid = valid_from_tree(cfg)
    g, _ = gpu_forward(cfg, inp, valid)
    P = oracle_params(cfg)
    tol = TOL[cfg.dtype]
    ndiff = 0
    for b in range(cfg.batch):
        for h in range(cfg.heads):
            ndiff += _check_head(cfg, inp, valid, g, b, h, P, tol)
    print(f"tie-justified index differences: {ndiff} rows")


def test_forward_scaling_sampled():
    """The 65536-point workload at full size; oracle on 96 sampled groups of two heads."""
    cfg = CONFIGS[3]
    print("forward parity config 3 (sampled)", flush=True)
    inp = make_inputs(cfg, layout="ball", with_grad=False)
    valid = valid_from_tree(cfg)
    g, _ = gpu_forward(cfg, inp, valid)
    P = oracle_params(cfg)
    rng = np.random.default_rng(3)
    ngroups = cfg.n_pad // cfg.group
    for h in (0, cfg.heads - 1):
        groups = np.sort(np.concatenate([[0, ngroups - 1], rng.choice(ngroups, 94, replace=False)]))
        groups = np.unique(groups)
        _check_head(cfg, inp, valid, g, 0, h, P, TOL[cfg.dtype], groups=groups)


def test_forward_no_own_ball_mask_and_mean_pool():
    cfg = CONFIGS[1]
    inp = make_inputs(cfg, layout="ball", with_grad=False)
    valid = np.ones((1, cfg.n_pad), bool)
    valid[0, 100:140] = False
    for kw, okw in ((dict(mask_own_ball=0), dict(mask_own_ball=False)), (dict(kv_pool=1), dict(kv_pool="mean"))):
        print(f"forward variant {kw}", flush=True)
        g, _ = gpu_forward(cfg, inp, valid, **kw)
        P = oracle_params(cfg, **okw)
        for h in range(cfg.heads):
            _check_head(cfg, inp, valid, g, 0, h, P, TOL[cfg.dtype])


@pytest.mark.parametrize("dtype,padded", [("bf16", False), ("f32", False), ("bf16", True)])
def test_forward_rising_maxima(dtype, padded):
    """Scores that rise along the key order by more than the lazy-rescale margin (8 in
    log2 units) in every 64-key tile, so the running maximum of the ball and compressed
    forward moves in each tile (O and row sums rescaled, prescaled scores shifted) instead
    of settling after the first tiles as on random data (the premise is checked on the
    CPU: test_host). A layer of 8192 points and two heads (bf16 unpadded: the shared
    forward launch, whole tiles; f32: the register-staged kernels; bf16 padded, every 97th
    slot a dummy: the masked kernels on two streams); mean pooling, so that the
    compressed keys are block means and rise with the keys. Scores stay within 52 log2
    units, where the compressed keys' bf16 storage moves a log-sum-exp by at most 0.008
    (float64 on the same inputs), inside the bf16 bar."""
    cfg = rising_config(dtype)
    print(f"forward parity, rising maxima (8192 points, 2 heads, {dtype}, padded={padded})", flush=True)
    inp = rising_inputs(cfg)
    valid = np.ones((1, cfg.n_pad), bool)
    if padded:
        valid[0, np.arange(cfg.n_pad) % 97 == 5] = False
    g, _ = gpu_forward(cfg, inp, valid, kv_pool=1)
    P = oracle_params(cfg, kv_pool="mean")
    for h in range(cfg.heads):
        _check_head(cfg, inp, valid, g, 0, h, P, TOL[cfg.dtype])


@pytest.mark.timeout(900)
def test_forward_large_full_shape():
    """The large workload at its stated shape: one cloud of 2^20 points (every slot real),
    16 heads of dim 64 (Q, K, V 2.1 GB each in bf16), ball 512, compression blocks of 32,
    selection blocks of 64, top-16, groups of 32, launched as the forward bench launches it.
    Inputs are drawn head by head (HeadInputs) and uploaded as they come. The oracle checks
    48 sampled groups (and every row of them) of three heads, incl. the first and last."""
    import torch

    from paper_2506_12541_amd import bsa as gb
    from parity import to_dev
    from workloads import HeadInputs

    cfg = CONFIGS[4]
    H, N, d = cfg.heads, cfg.n_pad, cfg.head_dim
    print("forward parity 2^20 points, 16 heads: drawing inputs", flush=True)
    hi = HeadInputs(cfg)
    p = gb.Params.from_config(cfg)
    q, k, v = (torch.empty((1, H, N, d), dtype=torch.bfloat16, device="cuda") for _ in range(3))
    checked = (0, 7, H - 1)
    host = {}

    def put(h, x):
        for name, t in (("q", q), ("k", k), ("v", v)):
            t[0, h].copy_(torch.from_numpy(x[name]).to("cuda").to(torch.bfloat16))
        if h in checked:
            host[h] = x

    hi.heads(put)
    gate = to_dev(hi.gate, torch.float32)
    phi_k = {w: to_dev(a, torch.float32) for w, a in hi.phi_k.items()}
    phi_v = {w: to_dev(a, torch.float32) for w, a in hi.phi_v.items()}
    print("forward parity 2^20 points, 16 heads: running the layer", flush=True)
    o, saved = gb.forward(p, q, k, v, None, gate, phi_k, phi_v)
    torch.cuda.synchronize()
    P = oracle_params(cfg)
    valid = np.ones((1, N), bool)
    rng = np.random.default_rng(4)
    ngroups = N // cfg.group
    for h in checked:
        print(f"forward parity 2^20 points: oracle on head {h}", flush=True)
        one = lambda t: t[None, None]
        g = {"o": one(o[0, h].float().cpu().numpy()),
             "o_branch": torch.stack([saved.o_branch[0, 0, h].float(), saved.o_cmp[0, h],
                                      saved.o_branch[1, 0, h].float()]).cpu().numpy()[:, None, None],
             "lse": saved.lse[:, 0, h].cpu().numpy()[:, None, None],
             "sel": one(saved.sel_idx[0, h].cpu().numpy().astype(np.int64)),
             "kc": one(saved.kcmp[0, h].cpu().numpy()), "vc": one(saved.vcmp[0, h].cpu().numpy())}
        inp = {n: one(host[h][n]) for n in ("q", "k", "v")}
        inp.update(gate=hi.gate, phi_k=hi.phi_k, phi_v=hi.phi_v)
        groups = np.unique(np.concatenate([[0, ngroups - 1], rng.choice(ngroups, 46, replace=False)]))
        _check_head(cfg, inp, valid, g, 0, 0, P, TOL[cfg.dtype], groups=groups)
