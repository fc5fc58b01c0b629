"""Pins for the block oracle (CPU only).

  * bfloat16 rounding against torch's float32 -> bfloat16 conversion (round to nearest
    even), ties included;
  * the block without rounding against a separate torch float64 formulation: RMSNorm from
    torch.nn.functional.rms_norm, linear maps from F.linear, silu from F.silu, the BSA layer
    as the dense masked-softmax formulation of the backward pins; torch autograd gives every
    gradient. The top-k selection is held at the oracle's (it has no gradient);
  * central finite differences of sum(y * dy) on the oracle's own forward;
  * the rounding reading: every stored bfloat16 tensor is representable, padding rows stay
    zero, and the rounded block stays within bfloat16 error of the unrounded one.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import bsa, model
from oracle.bsa import Params
from test_oracle_backward import dense_layer_torch

H, D = 2, 8
C = H * D
FF = 4 * C


def _setup(seed, P, B=2, n=64, n_real=53):
    rng = np.random.default_rng(seed)
    valid = np.zeros((B, n), bool)
    for b in range(B):
        valid[b, rng.choice(n, n_real, replace=False)] = True
    r = lambda *s: rng.standard_normal(s)
    x = r(B, n, C) * valid[..., None]
    W = {"g1": 1 + 0.1 * r(C), "wqkv": r(3 * C, C) / C ** 0.5, "wg": r(3, C) / C ** 0.5,
         "wo": r(C, C) / C ** 0.5, "g2": 1 + 0.1 * r(C), "w1": r(FF, C) / C ** 0.5,
         "w3": r(FF, C) / C ** 0.5, "w2": r(C, FF) / FF ** 0.5}
    phi = lambda: {"w1": r(P.cmp_block * D, D) * 0.2, "b1": r(D) * 0.2, "w2": r(D, D) * 0.2,
                   "b2": r(D) * 0.2}
    return dict(P=P, x=x, valid=valid, W=W, phi_k=phi(), phi_v=phi(), phi_q=phi(), dy=r(B, n, C))


PARAMS = [Params(ball=16, cmp_block=4, slc_block=8, topk=2, group=4),
          Params(ball=16, cmp_block=4, slc_block=8, topk=2, group=4, q_coarsen="mlp", group_compression=True)]
IDS = ["regular", "mlp_coarsen+group_cmp"]


def _oracle(s, bf16=False, sel=None):
    y, cache = model.block_forward(s["x"], s["valid"], s["W"], s["phi_k"], s["phi_v"], s["P"], H, D, sel=sel,
                                   phi_q=s["phi_q"], bf16=bf16)
    return y, cache


def test_round_bf16_matches_torch():
    rng = np.random.default_rng(0)
    x = (rng.standard_normal(20000) * np.exp(rng.uniform(-20, 20, 20000))).astype(np.float32)
    # exact halfway cases between neighbouring bfloat16 values: ties go to the even mantissa
    base = torch.from_numpy(rng.standard_normal(2000).astype(np.float32)).to(torch.bfloat16).float().numpy()
    bits = base.view(np.uint32) + np.uint32(0x8000)           # + half a bfloat16 ulp
    x = np.concatenate([x, bits.view(np.float32), -bits.view(np.float32), [0.0, 1.0, -2.5]]).astype(np.float32)
    ref = torch.from_numpy(x).to(torch.bfloat16).double().numpy()
    np.testing.assert_array_equal(model.round_bf16(x.astype(np.float64)), ref)


def _torch_block(s, sel):
    P = s["P"]
    t = lambda a: torch.tensor(a, dtype=torch.float64, requires_grad=True)
    x = t(s["x"])
    W = {k: t(v) for k, v in s["W"].items()}
    pk, pv, pq = ({w: t(a) for w, a in s[n].items()} for n in ("phi_k", "phi_v", "phi_q"))
    valid = torch.from_numpy(s["valid"])
    B, n, _ = x.shape
    xn1 = F.rms_norm(x, (C,), W["g1"], eps=model.EPS)
    qkv = F.linear(xn1, W["wqkv"])
    heads = lambda z: z.reshape(B, n, H, D).permute(0, 2, 1, 3)
    q, k, v = heads(qkv[..., :C]), heads(qkv[..., C:2 * C]), heads(qkv[..., 2 * C:])
    gate = F.linear(xn1, W["wg"])
    o = dense_layer_torch(q, k, v, valid, gate, pk, pv, pq, P, sel)
    h = x + F.linear(o.permute(0, 2, 1, 3).reshape(B, n, C), W["wo"])
    xn2 = F.rms_norm(h, (C,), W["g2"], eps=model.EPS)
    y = h + F.linear(F.silu(F.linear(xn2, W["w1"])) * F.linear(xn2, W["w3"]), W["w2"])
    (y * torch.from_numpy(s["dy"])).sum().backward()
    gr = lambda z: z.grad.numpy() if z.grad is not None else None
    return y.detach().numpy(), gr(x), {k: gr(v) for k, v in W.items()}, \
        {w: gr(a) for w, a in pk.items()}, {w: gr(a) for w, a in pv.items()}, {w: gr(a) for w, a in pq.items()}


@pytest.mark.parametrize("P", PARAMS, ids=IDS)
def test_block_matches_torch_autograd(P):
    s = _setup(1, P)
    y, cache = _oracle(s)
    gb = model.block_backward(s["dy"], cache, s["valid"], s["phi_k"], s["phi_v"], P, H, D, phi_q=s["phi_q"])
    ty, tdx, tdW, tpk, tpv, tpq = _torch_block(s, cache["fwd"]["sel"])
    close = lambda a, b: np.testing.assert_allclose(a, b, rtol=1e-9, atol=1e-11)
    close(y, ty)
    close(gb["dx"], tdx)
    for k in model.WEIGHTS:
        close(gb["dW"][k], tdW[k])
    for w in tpk:
        close(gb["dphi_k"][w], tpk[w])
        close(gb["dphi_v"][w], tpv[w])
        if P.group_compression:
            close(gb["dphi_q"][w], tpq[w])


def test_block_finite_differences():
    P = PARAMS[0]
    s = _setup(2, P)
    y, cache = _oracle(s)
    sel = cache["fwd"]["sel"]
    gb = model.block_backward(s["dy"], cache, s["valid"], s["phi_k"], s["phi_v"], P, H, D)
    loss = lambda: float(np.sum(_oracle(s, sel=sel)[0] * s["dy"]))
    rng = np.random.default_rng(3)
    eps = 1e-6
    real = np.argwhere(s["valid"])
    for name in ("x",) + model.WEIGHTS:
        arr = s["x"] if name == "x" else s["W"][name]
        grad = gb["dx"] if name == "x" else gb["dW"][name]
        for _ in range(3):
            if name == "x":
                b, i = real[rng.integers(len(real))]
                idx = (b, i, rng.integers(C))
            else:
                idx = tuple(rng.integers(sz) for sz in arr.shape)
            old = arr[idx]
            arr[idx] = old + eps
            lp = loss()
            arr[idx] = old - eps
            lm = loss()
            arr[idx] = old
            fd = (lp - lm) / (2 * eps)
            assert abs(fd - grad[idx]) < 1e-6 * max(1.0, abs(fd)), (name, idx, fd, grad[idx])


@pytest.mark.parametrize("P", PARAMS, ids=IDS)
def test_rounding_reading(P):
    s = _setup(4, P)
    y0, c0 = _oracle(s)
    sel = c0["fwd"]["sel"]
    y1, c1 = _oracle(s, bf16=True, sel=sel)
    for name in ("x1", "q", "k", "v", "om", "x2", "u", "w", "a"):
        np.testing.assert_array_equal(model.round_bf16(c1[name]), c1[name], err_msg=name)
    pad = ~s["valid"]
    assert not np.any(y1[pad]) and not np.any(c1["h"][pad])
    # relative to the magnitude of each row: a few bfloat16 steps of error after two sublayers
    scale = np.abs(y0).max()
    assert np.abs(y1 - y0).max() < 0.05 * scale
    g0 = model.block_backward(s["dy"], c0, s["valid"], s["phi_k"], s["phi_v"], P, H, D, phi_q=s["phi_q"])
    g1 = model.block_backward(s["dy"], c1, s["valid"], s["phi_k"], s["phi_v"], P, H, D, phi_q=s["phi_q"])
    np.testing.assert_array_equal(model.round_bf16(g1["do"]), g1["do"])
    for k in model.WEIGHTS:
        err = np.abs(g1["dW"][k] - g0["dW"][k]).max()
        assert err < 0.05 * g0["abs"][k].max(), k
    assert np.abs(g1["dx"] - g0["dx"]).max() < 0.05 * np.abs(g0["dx"]).max()
