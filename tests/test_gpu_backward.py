"""GPU backward pass vs the float64 oracle's analytic gradients on the same inputs.

The oracle runs with the GPU's selected blocks (ties within 1e-6 may pick different
blocks; the gradient is defined for a fixed selection). dQ, dK, dV are compared by
max-abs error; weight and gate-logit gradients, which are sums over many terms, by the
error of each entry relative to the magnitude of its summed terms (sum of |term|, the
standard error bound of a sum; the bias of the key MLP's last layer has an identically
zero gradient because a shift of every compressed key leaves each softmax unchanged).
Bar: 1e-4 (f32) / 2e-2 (bf16)."""
import numpy as np
import pytest
import torch

from oracle import bsa as ob
from parity import TOL, gpu_forward, max_abs, oracle_kw, oracle_params, to_dev, valid_from_tree
from paper_2506_12541_amd import bsa as gb
from workloads import CONFIGS, Config, make_inputs, round_bf16

pytestmark = pytest.mark.gpu


def oracle_with_sel(inp, valid, P, sel):
    """Oracle forward caches, with the selection branch re-run on the given blocks."""
    f64 = lambda a: np.asarray(a, np.float64)
    q, k, v = f64(inp["q"]), f64(inp["k"]), f64(inp["v"])
    fwd = ob.forward(q, k, v, valid, inp["gate"], inp["phi_k"], inp["phi_v"], P, phi_q=inp.get("phi_q"))
    fwd["sel"] = sel
    B, H = q.shape[:2]
    for b in range(B):
        for h in range(H):
            fwd["o_branch"][2, b, h], fwd["lse"][2, b, h] = ob.selection_branch(q[b, h], k[b, h], v[b, h], valid[b],
                                                                                sel[b, h], P)
    return fwd


def run_case(cfg, seed=None, gate_scale=1.0, inp=None, **pkw):
    inp = make_inputs(cfg, seed, layout="ball", with_grad=True) if inp is None else inp
    inp["gate"] = (inp["gate"] * gate_scale).astype(np.float32)
    valid = valid_from_tree(cfg)
    g, (p, q, k, v, vd, gate, phi_k, phi_v, saved, o, phi_q) = gpu_forward(cfg, inp, valid, **pkw)
    dout = to_dev(inp["do"], p.torch_dtype)
    grads = gb.backward(p, q, k, v, vd, gate, phi_k, phi_v, saved, dout, phi_q=phi_q)
    torch.cuda.synchronize()
    P = oracle_params(cfg, **oracle_kw(pkw))
    fwd = oracle_with_sel(inp, valid, P, g["sel"])
    ref = ob.backward(inp["q"], inp["k"], inp["v"], valid, inp["gate"], inp["phi_k"], inp["phi_v"], P, fwd, inp["do"],
                      phi_q=inp["phi_q"])
    tol = TOL[cfg.dtype]
    out = {n: grads[n].cpu().numpy() for n in ("dq", "dk", "dv", "dgate")}
    errs = {}
    for n in ("dq", "dk", "dv"):
        errs[n] = max_abs(out[n], ref[n])
    # summed gradients: |gpu - oracle| relative to the magnitude of the summed terms
    rel = lambda g, r, a: float(np.max(np.abs(np.asarray(g, np.float64) - r) / np.maximum(a, 1e-30)))
    errs["dgate"] = rel(out["dgate"], ref["dgate"], ref["abs"]["dgate"])
    mlps = ("dphi_k", "dphi_v") if P.kv_pool == "mlp" else ()
    if P.group_compression and P.q_coarsen == "mlp":
        mlps += ("dphi_q",)
    zero = {}
    for which in mlps:
        for w in ("w1", "b1", "w2", "b2"):
            gw = grads[which][w].cpu().numpy()
            if ref["abs"][which][w].max() < 1e-12:
                # every term of the oracle's sum vanishes: the gradient is identically zero
                # (a softmax over one eligible compressed key is constant, so dK^ = 0), and
                # the GPU's value is float32 rounding of dP - D, bounded absolutely
                zero[f"{which}.{w}"] = float(np.abs(gw).max())
            else:
                errs[f"{which}.{w}"] = rel(gw, ref[which][w], ref["abs"][which][w])
    print({k: f"{v:.2e}" for k, v in errs.items()}, {k: f"|{v:.1e}|" for k, v in zero.items()}, flush=True)
    bad = {k: v for k, v in errs.items() if not v < tol}
    bad.update({k: v for k, v in zero.items() if not v < 1e-6})
    assert not bad, bad
    # padding slots carry no gradient
    for n in ("dq", "dk", "dv"):
        for b in range(cfg.batch):
            assert not np.any(out[n][b][:, ~valid[b]])
    return g


def test_backward_tiny_fp32():
    print("backward parity config 1", flush=True)
    run_case(CONFIGS[1])


def test_backward_tiny_fp32_isolated_branches():
    # saturated gates isolate each branch (sigmoid(+-12) ~ 1 / 6e-6)
    cfg = CONFIGS[1]
    for scale in (30.0,):
        print(f"backward parity config 1, gate scale {scale}", flush=True)
        run_case(cfg, gate_scale=scale)


def test_backward_airflow_bf16():
    print("backward parity config 5", flush=True)
    run_case(CONFIGS[5])


def test_backward_variants():
    cfg = CONFIGS[1]
    for kw in (dict(mask_own_ball=0), dict(kv_pool=1)):
        print(f"backward variant {kw}", flush=True)
        run_case(cfg, **kw)


def test_backward_small_bf16_with_padding():
    cfg = Config("small_bf16", 2, 900, 1024, 2, 64, "bf16", 128, 16, 16, 32, 4, 16, "uniform", "fwdbwd")
    print("backward parity small bf16 d=64", flush=True)
    run_case(cfg, seed=11)


def test_backward_heavily_selected_block():
    """One selection block chosen by every query group outside its ball (its keys and every
    query share a strong common direction; mean-pooled compressed keys keep that direction),
    so its item list exceeds the one-wave limit of the selection dK/dV pass and takes the
    pass's heavy-block path; l' = 32 (eight waves per heavy block) and l' = 64 (four)."""
    for ls in (32, 64):
        cfg = Config(f"heavy_block_ls{ls}", 1, 8192, 8192, 2, 64, "bf16", 256, 16, 16, ls, 4, 16, "uniform", "fwdbwd")
        inp = make_inputs(cfg, 7, layout="ball", with_grad=True)
        u = np.zeros(cfg.head_dim)
        u[::2] = 1.0 / np.sqrt(cfg.head_dim / 2)
        hot = 77                                          # the selection block everyone chooses
        # (kept representable in bfloat16, as the generator's inputs are)
        inp["q"] = round_bf16(inp["q"] + 2.0 * u).astype(inp["q"].dtype)
        k = inp["k"].astype(np.float64)
        k[:, :, hot * ls:(hot + 1) * ls] += 4.0 * u
        inp["k"] = round_bf16(k).astype(inp["k"].dtype)
        print(f"backward parity, heavily selected block, l' = {ls}", flush=True)
        g = run_case(cfg, inp=inp, kv_pool=1)
        sel = g["sel"]
        most = max(int(np.bincount(sel[0, h][sel[0, h] >= 0].ravel()).max()) for h in range(cfg.heads))
        print("most items in one block:", most, flush=True)
        assert most > 256, most


def test_backward_scaling_one_head():
    """65536 points, 8 heads, d=64 at full size (the benchmarked workload); the oracle
    differentiates one whole head (heads are independent except for the gate and MLP
    weight gradients, which sum over heads and are checked on the airflow workload)."""
    cfg = CONFIGS[3]
    print("backward parity config 3 (head 5)", flush=True)
    inp = make_inputs(cfg, layout="ball", with_grad=True)
    valid = valid_from_tree(cfg)
    g, (p, q, k, v, vd, gate, phi_k, phi_v, saved, o, _) = gpu_forward(cfg, inp, valid)
    grads = gb.backward(p, q, k, v, vd, gate, phi_k, phi_v, saved, to_dev(inp["do"], p.torch_dtype))
    torch.cuda.synchronize()
    h = 5
    one = {n: np.ascontiguousarray(inp[n][:, h:h + 1]) for n in ("q", "k", "v", "do")}
    one.update(gate=inp["gate"], phi_k=inp["phi_k"], phi_v=inp["phi_v"])
    P = oracle_params(cfg)
    fwd = oracle_with_sel(one, valid, P, g["sel"][:, h:h + 1])
    ref = ob.backward(one["q"], one["k"], one["v"], valid, one["gate"], one["phi_k"], one["phi_v"], P, fwd,
                      one["do"])
    errs = {n: max_abs(grads[n][:, h:h + 1].cpu().numpy(), ref[n]) for n in ("dq", "dk", "dv")}
    print({k: f"{v:.2e}" for k, v in errs.items()}, flush=True)
    assert all(e < TOL[cfg.dtype] for e in errs.values()), errs


def test_backward_scaling_group_compression_one_head():
    """The 65536-point workload with MLP query coarsening and group compression (Eq. 13-15),
    one head against the oracle. Its selection concentrates on a few blocks (one block is
    chosen by about a thousand groups), so the selection dK/dV pass takes its path for
    blocks with many items (more than 256 (group, query-block) items: eight waves per
    block); the test checks that such a block is present."""
    cfg = CONFIGS[3]
    pkw = dict(q_coarsen=1, group_compression=1)
    print("backward parity config 3, group compression (head 2)", flush=True)
    inp = make_inputs(cfg, layout="ball", with_grad=True)
    valid = valid_from_tree(cfg)
    g, (p, q, k, v, vd, gate, phi_k, phi_v, saved, o, phi_q) = gpu_forward(cfg, inp, valid, **pkw)
    grads = gb.backward(p, q, k, v, vd, gate, phi_k, phi_v, saved, to_dev(inp["do"], p.torch_dtype), phi_q=phi_q)
    torch.cuda.synchronize()
    h = 2
    sel = g["sel"][:, h:h + 1]
    counts = np.bincount(sel[sel >= 0].ravel(), minlength=cfg.n_pad // cfg.slc_block)
    assert counts.max() > 256, counts.max()
    one = {n: np.ascontiguousarray(inp[n][:, h:h + 1]) for n in ("q", "k", "v", "do")}
    one.update(gate=inp["gate"], phi_k=inp["phi_k"], phi_v=inp["phi_v"], phi_q=inp["phi_q"])
    P = oracle_params(cfg, **oracle_kw(pkw))
    fwd = oracle_with_sel(one, valid, P, sel)
    ref = ob.backward(one["q"], one["k"], one["v"], valid, one["gate"], one["phi_k"], one["phi_v"], P, fwd,
                      one["do"], phi_q=one["phi_q"])
    errs = {n: max_abs(grads[n][:, h:h + 1].cpu().numpy(), ref[n]) for n in ("dq", "dk", "dv")}
    print({k: f"{v:.2e}" for k, v in errs.items()}, "most items in one block:", int(counts.max()), flush=True)
    assert all(e < TOL[cfg.dtype] for e in errs.values()), errs


def test_one_stream_equals_two_streams():
    """Every kernel is deterministic and the two-stream schedule only reorders independent
    branches, so one-stream and two-stream runs give bit-identical results."""
    cfg = Config("small_bf16", 2, 900, 1024, 2, 64, "bf16", 128, 16, 16, 32, 4, 16, "uniform", "fwdbwd")
    from paper_2506_12541_amd import _lib
    lib = _lib.load()
    inp = make_inputs(cfg, 11, layout="ball", with_grad=True)
    valid = valid_from_tree(cfg)
    outs = []
    try:
        for n in (2, 1):
            _lib.check(lib.bsa_set_streams(n), "streams")
            g, (p, q, k, v, vd, gate, phi_k, phi_v, saved, o, phi_q) = gpu_forward(cfg, inp, valid)
            grads = gb.backward(p, q, k, v, vd, gate, phi_k, phi_v, saved, to_dev(inp["do"], p.torch_dtype))
            torch.cuda.synchronize()
            outs.append((o.clone(), {n_: grads[n_].clone() for n_ in ("dq", "dk", "dv", "dgate")}))
    finally:
        lib.bsa_set_streams(2)
    assert torch.equal(outs[0][0], outs[1][0])
    for n_ in ("dq", "dk", "dv", "dgate"):
        assert torch.equal(outs[0][1][n_], outs[1][1][n_]), n_
