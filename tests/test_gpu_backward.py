"""GPU backward pass vs the float64 oracle's analytic gradients on the same inputs.

The oracle runs with the GPU's selected blocks (ties within 1e-6 may pick different
blocks; the gradient is defined for a fixed selection). dQ, dK, dV are compared by
max-abs error; weight and gate-logit gradients, which are sums over many terms, by
max |gpu - oracle| / max |oracle| (tests/bars.py: a zeroed or sign-flipped gradient
fails; the key MLP's output bias, identically zero by the softmax's shift invariance, is
bounded by its summed-term magnitude). Bar: 1e-4 (f32) / 2e-2 (bf16)."""
import dataclasses

import numpy as np
import pytest
import torch

from oracle import bsa as ob
from bars import check_summed, oracle_summed
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


def check_layer_summed(grads, ref, P, tol):
    """Gate-logit and MLP weight gradients of the layer against the oracle's (bars.py)."""
    mlps = ("dphi_k", "dphi_v") if P.kv_pool == "mlp" else ()
    if P.group_compression and P.q_coarsen == "mlp":
        mlps += ("dphi_q",)
    flat = oracle_summed(ref, mlps)
    got = {"dgate": grads["dgate"].cpu().numpy()}
    for m in mlps:
        for w in ("w1", "b1", "w2", "b2"):
            got[f"{m}.{w}"] = grads[m][w].cpu().numpy()
    return check_summed(got, flat, tol)


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
    errs = {n: max_abs(out[n], ref[n]) for n in ("dq", "dk", "dv")}
    print({k: f"{v:.2e}" for k, v in errs.items()}, flush=True)
    assert all(e < tol for e in errs.values()), errs
    check_layer_summed(grads, ref, P, tol)
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


@pytest.mark.parametrize("store_lse", [1, 0])
def test_backward_airflow_bf16(store_lse):
    """Config 5 with the per-branch softmax statistics stored by the forward pass (1) or
    recomputed by the backward pass (0)."""
    print(f"backward parity config 5, store_lse={store_lse}", flush=True)
    run_case(CONFIGS[5], store_lse=store_lse)


SMALL_BF16 = Config("small_bf16", 2, 900, 1024, 2, 64, "bf16", 128, 16, 16, 32, 4, 16, "uniform", "fwdbwd")


@pytest.mark.parametrize("case", ["tiny_fp32", "small_bf16", "group_compression", "per_token", "mean_pool"])
def test_recomputed_lse_gives_identical_gradients(case):
    """store_lse = 0 recomputes each branch's log-sum-exp rows with the forward kernels minus
    the value products (same tiles and order), so every gradient equals the store_lse = 1
    run bit for bit; the recompute-mode gradients are also checked against the oracle."""
    cfg, seed, pkw = {
        "tiny_fp32": (CONFIGS[1], None, {}),
        "small_bf16": (SMALL_BF16, 11, {}),
        "group_compression": (SMALL_BF16, 12, dict(q_coarsen=1, group_compression=1)),
        "per_token": (dataclasses.replace(SMALL_BF16, group=1), 13, {}),
        "mean_pool": (SMALL_BF16, 14, dict(kv_pool=1)),
    }[case]
    inp = make_inputs(cfg, seed, layout="ball", with_grad=True)
    valid = valid_from_tree(cfg)
    outs = []
    for store in (1, 0):
        g, (p, q, k, v, vd, gate, phi_k, phi_v, saved, o, phi_q) = gpu_forward(cfg, inp, valid, store_lse=store,
                                                                               **pkw)
        assert (saved.lse is None) == (store == 0)
        grads = gb.backward(p, q, k, v, vd, gate, phi_k, phi_v, saved, to_dev(inp["do"], p.torch_dtype), phi_q=phi_q)
        torch.cuda.synchronize()
        flat = {n: grads[n].clone() for n in ("dq", "dk", "dv", "dgate")}
        for m in ("dphi_k", "dphi_v", "dphi_q"):
            flat.update({f"{m}.{w}": t.clone() for w, t in grads[m].items()})
        outs.append((o.clone(), flat))
    print(f"recompute-LSE case {case}: {len(outs[0][1])} gradients", flush=True)
    assert torch.equal(outs[0][0], outs[1][0])
    for n in outs[0][1]:
        assert torch.equal(outs[0][1][n], outs[1][1][n]), n
    run_case(cfg, seed=seed, store_lse=0, **pkw)


@pytest.mark.timeout(600)
def test_recomputed_lse_identical_at_scaling_shape():
    """The benchmarked shape (65536 points, H=8, d=64, bf16): store_lse = 0 gives the
    gradients of store_lse = 1 bit for bit (both against the oracle at this size are covered
    by test_backward_scaling_all_heads)."""
    cfg = CONFIGS[3]
    inp = make_inputs(cfg, layout="ball", with_grad=True)
    valid = valid_from_tree(cfg)
    outs = []
    for store in (1, 0):
        print(f"recompute-LSE at 65536 points, store_lse={store}", flush=True)
        g, (p, q, k, v, vd, gate, phi_k, phi_v, saved, o, phi_q) = gpu_forward(cfg, inp, valid, store_lse=store)
        grads = gb.backward(p, q, k, v, vd, gate, phi_k, phi_v, saved, to_dev(inp["do"], p.torch_dtype))
        torch.cuda.synchronize()
        flat = {n: grads[n].clone() for n in ("dq", "dk", "dv", "dgate")}
        for m in ("dphi_k", "dphi_v"):
            flat.update({f"{m}.{w}": t.clone() for w, t in grads[m].items()})
        outs.append((o.clone(), flat))
        del g, saved, grads
    assert torch.equal(outs[0][0], outs[1][0])
    for n in outs[0][1]:
        assert torch.equal(outs[0][1][n], outs[1][1][n]), n


def test_backward_variants():
    cfg = CONFIGS[1]
    for kw in (dict(mask_own_ball=0), dict(kv_pool=1)):
        print(f"backward variant {kw}", flush=True)
        run_case(cfg, **kw)


def test_backward_full_clouds_unmasked():
    """Clouds with no padding launch without a mask, as the benchmark does: the unmasked
    kernels and the shared launches (ball and compressed forward; their key-major passes)."""
    run_case(Config("full_bf16", 2, 2048, 2048, 2, 64, "bf16", 128, 16, 16, 32, 4, 16, "uniform", "fwdbwd"), seed=21)


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


@pytest.mark.timeout(600)
def test_backward_scaling_all_heads():
    """65536 points, 8 heads, d=64 at full size (the benchmarked workload, launched as the
    benchmark launches it): the oracle differentiates the whole layer, so every dQ, dK, dV
    entry and the gate-logit and MLP weight gradients (sums over all heads and 4096
    compressed blocks per head) are compared."""
    cfg = CONFIGS[3]
    print("backward parity config 3 (all heads)", flush=True)
    inp = make_inputs(cfg, layout="ball", with_grad=True)
    valid = valid_from_tree(cfg)
    g, (p, q, k, v, vd, gate, phi_k, phi_v, saved, o, _) = gpu_forward(cfg, inp, valid)
    grads = gb.backward(p, q, k, v, vd, gate, phi_k, phi_v, saved, to_dev(inp["do"], p.torch_dtype))
    torch.cuda.synchronize()
    P = oracle_params(cfg)
    fwd = oracle_with_sel(inp, valid, P, g["sel"])
    print("oracle forward done", flush=True)
    ref = ob.backward(inp["q"], inp["k"], inp["v"], valid, inp["gate"], inp["phi_k"], inp["phi_v"], P, fwd,
                      inp["do"])
    tol = TOL[cfg.dtype]
    errs = {n: max_abs(grads[n].cpu().numpy(), ref[n]) for n in ("dq", "dk", "dv")}
    print({k: f"{v:.2e}" for k, v in errs.items()}, flush=True)
    assert all(e < tol for e in errs.values()), errs
    check_layer_summed(grads, ref, P, tol)


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


@pytest.mark.parametrize("full", [False, True])
def test_one_stream_equals_two_streams(full):
    """Every kernel is deterministic and the two-stream schedule only reorders independent
    branches, so one-stream and two-stream runs give bit-identical results; so do runs
    without the shared launches (streams mode 0: the ball and compressed forward, and their
    key-major backward passes, each in launches of their own). full: 2048-point clouds with
    no padding (no mask: the shared launches run in modes 1 and 2)."""
    cfg = Config("small_bf16", 2, 900, 1024, 2, 64, "bf16", 128, 16, 16, 32, 4, 16, "uniform", "fwdbwd")
    if full:
        cfg = Config("full_bf16", 2, 2048, 2048, 2, 64, "bf16", 128, 16, 16, 32, 4, 16, "uniform", "fwdbwd")
    from paper_2506_12541_amd import _lib
    lib = _lib.load()
    inp = make_inputs(cfg, 11, layout="ball", with_grad=True)
    valid = valid_from_tree(cfg)
    outs = []
    try:
        for n in (2, 1, 0):
            _lib.check(lib.bsa_set_streams(n), "streams")
            g, (p, q, k, v, vd, gate, phi_k, phi_v, saved, o, phi_q) = gpu_forward(cfg, inp, valid)
            grads = gb.backward(p, q, k, v, vd, gate, phi_k, phi_v, saved, to_dev(inp["do"], p.torch_dtype))
            torch.cuda.synchronize()
            outs.append((o.clone(), {n_: grads[n_].clone() for n_ in ("dq", "dk", "dv", "dgate")}))
    finally:
        lib.bsa_set_streams(2)
    for other in outs[1:]:
        assert torch.equal(outs[0][0], other[0])
        for n_ in ("dq", "dk", "dv", "dgate"):
            assert torch.equal(outs[0][1][n_], other[1][n_]), n_
