"""One transformer block around the BSA layer, forward and backward, in float64 (oracle;
test infrastructure only: the product path never calls it).

The paper's model stacks 18 blocks, each holding an RMSNorm, a BSA layer and a SwiGLU
(Section 3.1, training details); it gives no block layout or sizes. Readings:
  * pre-norm residual block:  h = x + merge(BSA(Q, K, V)) W_o^T,  y = h + SwiGLU(norm2(h)),
    with Q, K, V and the gate logits of Eq. 9 taken from norm1(x);
  * RMSNorm(z) = z / sqrt(mean(z^2) + eps) * g, eps = 1e-6, one learned gain g [C] per norm;
  * bias-free linear maps stored as [out, in]: W_qkv [3C, C] (head h of Q uses output
    columns h d .. (h+1) d, then K, then V), W_g [3, C] (gate logits, ball / compression /
    selection), W_o [C, C];
  * SwiGLU(z) = (silu(z W_1^T) * (z W_3^T)) W_2^T with hidden size F (4C in the workloads)
    and silu(u) = u sigmoid(u); W_1, W_3 [F, C], W_2 [C, F];
  * padding slots hold zero rows; every map is bias-free, so they stay zero.

Precision reading (``bf16=True``), that of bf16 mixed-precision training: every matrix
product over the channels takes bfloat16 operands (round to nearest even) and accumulates
exactly; Q, K, V, the attention output, the SwiGLU pre-activations u, w and its output a are
stored in bfloat16; the residual stream, both norms, the gate logits (from the unrounded
norm1 output and W_g) and every gradient that leaves a product stay wide. In the backward
pass the gradients that enter a product (dy, the SwiGLU pre-activation gradients, dh, dO
and dQ/dK/dV) are rounded the same way. With ``bf16=False`` nothing is rounded.
The BSA layer is ``bsa.forward`` / ``bsa.backward`` (Q, K, V as [B, H, N, d]).
"""
from __future__ import annotations

import numpy as np

from . import bsa

EPS = 1e-6
WEIGHTS = ("g1", "wqkv", "wg", "wo", "g2", "w1", "w3", "w2")


def round_bf16(x):
    """Round to the nearest bfloat16 (8 significant bits, ties to even); values stay in
    the normal range of bfloat16 here, so the exponent is never clamped."""
    x = np.asarray(x, np.float64)
    m, e = np.frexp(x)                          # x = m 2^e, 0.5 <= |m| < 1
    return np.ldexp(np.round(m * 256.0) / 256.0, e)


def rmsnorm(x, g):
    r = 1.0 / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + EPS)
    return x * r * g, {"x": x, "r": r, "g": g}


def rmsnorm_backward(dy, c):
    """dx, and dg with the magnitudes of its summed terms."""
    x, r, g = c["x"], c["r"], c["g"]
    xhat = x * r
    dxhat = dy * g
    dx = r * (dxhat - xhat * np.mean(dxhat * xhat, axis=-1, keepdims=True))
    lead = tuple(range(dy.ndim - 1))
    return dx, np.sum(dy * xhat, axis=lead), np.sum(np.abs(dy * xhat), axis=lead)


def silu(u):
    return u * bsa.sigmoid(u)


def silu_grad(u):
    s = bsa.sigmoid(u)
    return s * (1.0 + u * (1.0 - s))


def split_heads(z, H, d):
    B, N, _ = z.shape
    return z.reshape(B, N, H, d).transpose(0, 2, 1, 3)


def merge_heads(z):
    B, H, N, d = z.shape
    return z.transpose(0, 2, 1, 3).reshape(B, N, H * d)


def _lin_grad(dy, x):
    """dW = dy^T x summed over all leading axes, and the sum of |terms|."""
    dy2, x2 = dy.reshape(-1, dy.shape[-1]), x.reshape(-1, x.shape[-1])
    return dy2.T @ x2, np.abs(dy2).T @ np.abs(x2)


def _rounder(bf16):
    return round_bf16 if bf16 else (lambda a: a)


def block_forward(x, valid, W, phi_k, phi_v, P: bsa.Params, H: int, d: int, sel=None, phi_q=None,
                  bf16=False):
    """y [B, N, C] and the caches of the backward pass. ``sel`` replaces the layer's own
    selection (the layer is then evaluated on the given blocks)."""
    rnd = _rounder(bf16)
    x = np.asarray(x, np.float64)
    W = {k: np.asarray(v, np.float64) for k, v in W.items()}
    Wr = {k: rnd(W[k]) for k in ("wqkv", "wo", "w1", "w3", "w2")}
    C = H * d
    xn1, c1 = rmsnorm(x, W["g1"])
    x1 = rnd(xn1)
    qkv = rnd(x1 @ Wr["wqkv"].T)
    q, k, v = (split_heads(qkv[..., i * C:(i + 1) * C], H, d) for i in range(3))
    gate = xn1 @ W["wg"].T
    fwd = bsa.forward(q, k, v, valid, gate, phi_k, phi_v, P, phi_q=phi_q)
    if sel is not None:
        fwd["sel"] = np.asarray(sel)
        for b in range(q.shape[0]):
            for hh in range(H):
                fwd["o_branch"][2, b, hh], fwd["lse"][2, b, hh] = bsa.selection_branch(
                    q[b, hh], k[b, hh], v[b, hh], valid[b], fwd["sel"][b, hh], P)
        sg = bsa.sigmoid(gate)
        fwd["o"] = sum(sg[:, None, :, br, None] * fwd["o_branch"][br] for br in range(3))
    om = rnd(merge_heads(fwd["o"]))
    h = x + om @ Wr["wo"].T
    xn2, c2 = rmsnorm(h, W["g2"])
    x2 = rnd(xn2)
    u = rnd(x2 @ Wr["w1"].T)
    w = rnd(x2 @ Wr["w3"].T)
    a = rnd(silu(u) * w)
    y = h + a @ Wr["w2"].T
    cache = dict(x=x, xn1=xn1, x1=x1, c1=c1, q=q, k=k, v=v, gate=gate, fwd=fwd, om=om, h=h, x2=x2,
                 c2=c2, u=u, w=w, a=a, W=W, Wr=Wr, bf16=bf16)
    return y, cache


def block_backward(dy, cache, valid, phi_k, phi_v, P: bsa.Params, H: int, d: int, phi_q=None):
    """Gradients of sum(y * dy): dx and every weight, with the magnitudes of the summed
    terms of each weight gradient (the error scale of a sum)."""
    rnd = _rounder(cache["bf16"])
    dy = np.asarray(dy, np.float64)
    W, Wr = cache["W"], cache["Wr"]
    g, gabs = {}, {}
    # SwiGLU sublayer
    dyr = rnd(dy)
    g["w2"], gabs["w2"] = _lin_grad(dyr, cache["a"])
    da = dyr @ Wr["w2"]
    u, w = cache["u"], cache["w"]
    du = rnd(da * w * silu_grad(u))
    dw = rnd(da * silu(u))
    g["w1"], gabs["w1"] = _lin_grad(du, cache["x2"])
    g["w3"], gabs["w3"] = _lin_grad(dw, cache["x2"])
    dxn2 = du @ Wr["w1"] + dw @ Wr["w3"]
    dh2, g["g2"], gabs["g2"] = rmsnorm_backward(dxn2, cache["c2"])
    dh = dy + dh2
    # attention sublayer
    dhr = rnd(dh)
    g["wo"], gabs["wo"] = _lin_grad(dhr, cache["om"])
    do = rnd(split_heads(dhr @ Wr["wo"], H, d))
    lb = bsa.backward(cache["q"], cache["k"], cache["v"], valid, cache["gate"], phi_k, phi_v, P, cache["fwd"],
                      do, phi_q=phi_q)
    dqkv = rnd(np.concatenate([merge_heads(lb["dq"]), merge_heads(lb["dk"]), merge_heads(lb["dv"])], axis=-1))
    g["wqkv"], gabs["wqkv"] = _lin_grad(dqkv, cache["x1"])
    g["wg"], gabs["wg"] = _lin_grad(lb["dgate"], cache["xn1"])
    dxn1 = dqkv @ Wr["wqkv"] + lb["dgate"] @ W["wg"]
    dx1, g["g1"], gabs["g1"] = rmsnorm_backward(dxn1, cache["c1"])
    dx = dh + dx1
    return {"dx": dx, "dW": g, "abs": gabs, "dphi_k": lb["dphi_k"], "dphi_v": lb["dphi_v"],
            "dphi_q": lb.get("dphi_q"), "do": do, "layer": lb}
