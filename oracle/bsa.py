"""Ball Sparse Attention layer, forward and backward, in float64 (oracle; tests only).

Inputs are in ball order (the output of the tree ordering): Q, K, V as [B, H, N, d],
``valid`` [B, N] (False for dummy slots), gate logits [B, N, 3] in branch order
(ball, compression, selection), and one compression MLP for keys and one for values,
each {w1 [l*d, d], b1 [d], w2 [d, d], b2 [d]}, shared across heads.

Readings of points the paper leaves open (each is stated where it is used):
  * attention bias B of Eq. 2 is zero; softmax scale 1/sqrt(d) in all three branches;
  * no causal mask anywhere (point sets are unordered, Section 1);
  * dummy slots are masked as keys, produce zero output rows as queries, and are zero
    rows inside a compressed block ("0-padded" in Eq. 5);
  * the MLP phi of Eq. 5 is l*d -> d -> d with exact-erf GELU and biases, applied to the
    token-major flatten of the block; a compressed token is a valid key iff its block
    holds at least one real token; mean pooling (also named by Eq. 5) divides by l;
  * importance scores are unscaled dot products (Eq. 6); the group form uses the pooled
    query of Eq. 11 over the group's real queries divided by g, which equals the group
    mean of Eq. 12 by linearity;
  * a selection block of l' = r*l tokens scores the mean of its r compressed-block
    scores; blocks inside the query group's own ball are excluded (Section 3.2,
    receptive-field paragraph), as are blocks with no real token;
  * top-k orders by (higher score, lower index); indices are stored ascending, padded
    with -1 when fewer than k* blocks are eligible;
  * the selection set is per head; the gate is per token and shared across heads;
  * a softmax row with no eligible key outputs zeros and has log-sum-exp -inf;
  * query coarsening (Eq. 13) pools blocks of l queries, so the selection groups of Eq.
    13-14 are those blocks (g = l); its MLP phi_q has the shape of phi_k, and its mean
    form is the pooled query of Eq. 11;
  * group compression (Eq. 15) attends from the coarse queries of Eq. 13 (a coarse query
    is valid iff its block holds a real token) and copies each result to the real
    queries of its block; dummy rows stay zero.
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np
from scipy.special import erf

NEG_INF = -np.inf


@dataclasses.dataclass(frozen=True)
class Params:
    ball: int                 # m, ball size (Eq. 3)
    cmp_block: int            # l, compression block length = stride (Eq. 5)
    slc_block: int            # l', selection block length (Eq. 8)
    topk: int                 # k*, number of selected blocks (Eq. 7)
    group: int                # g, query group size (Eq. 10)
    mask_own_ball: bool = True
    kv_pool: str = "mlp"      # "mlp" or "mean" (Eq. 5)
    scale: float | None = None
    q_coarsen: str = "mean"   # "mean" (Eq. 11) or "mlp" (phi_q of Eq. 13; needs g = l)
    group_compression: bool = False   # Eq. 15 (needs g = l)

    def __post_init__(self):
        if (self.q_coarsen == "mlp" or self.group_compression) and self.group != self.cmp_block:
            raise ValueError("query coarsening over blocks (Eq. 13, 15) needs group == cmp_block")

    def sm_scale(self, d: int) -> float:
        return 1.0 / math.sqrt(d) if self.scale is None else float(self.scale)


# ----------------------------------------------------------------------------------
# Scaled dot-product attention over an explicit key set (Eq. 2 with B = 0).
# ----------------------------------------------------------------------------------
def attend(q, k, v, key_valid, scale):
    """softmax(q k^T * scale) v over the keys with key_valid; returns (o, lse)."""
    nq = q.shape[0]
    o = np.zeros((nq, v.shape[1]))
    lse = np.full(nq, NEG_INF)
    if nq == 0 or not np.any(key_valid):
        return o, lse
    s = (q @ k[key_valid].T) * scale
    mx = s.max(axis=1, keepdims=True)
    p = np.exp(s - mx)
    den = p.sum(axis=1, keepdims=True)
    o = (p @ v[key_valid]) / den
    lse = mx[:, 0] + np.log(den[:, 0])
    return o, lse


def attend_backward(q, k, v, key_valid, scale, o, lse, do):
    """Gradients of attend() given the upstream gradient do of its output."""
    dq = np.zeros_like(q)
    dk = np.zeros_like(k)
    dv = np.zeros_like(v)
    if q.shape[0] == 0 or not np.any(key_valid):
        return dq, dk, dv
    kk, vv = k[key_valid], v[key_valid]
    s = (q @ kk.T) * scale
    p = np.exp(s - lse[:, None])
    dp = do @ vv.T
    delta = np.sum(do * o, axis=1, keepdims=True)
    ds = p * (dp - delta)
    dq = (ds @ kk) * scale
    dk[key_valid] = (ds.T @ q) * scale
    dv[key_valid] = p.T @ do
    return dq, dk, dv


# ----------------------------------------------------------------------------------
# Branch 1: Ball Tree Attention, attention inside each ball of m slots (Eq. 3).
# ----------------------------------------------------------------------------------
def ball_branch(q, k, v, valid, P: Params):
    n, d = q.shape
    m = P.ball
    o = np.zeros((n, d))
    lse = np.full(n, NEG_INF)
    for s in range(0, n, m):
        e = s + m
        rows = np.nonzero(valid[s:e])[0] + s
        oo, ll = attend(q[rows], k[s:e], v[s:e], valid[s:e], P.sm_scale(d))
        o[rows], lse[rows] = oo, ll
    return o, lse


def ball_branch_backward(q, k, v, valid, P: Params, o, lse, do):
    n, d = q.shape
    m = P.ball
    dq, dk, dv = np.zeros_like(q), np.zeros_like(k), np.zeros_like(v)
    for s in range(0, n, m):
        e = s + m
        rows = np.nonzero(valid[s:e])[0] + s
        gq, gk, gv = attend_backward(q[rows], k[s:e], v[s:e], valid[s:e], P.sm_scale(d),
                                     o[rows], lse[rows], do[rows])
        dq[rows] = gq
        dk[s:e] += gk
        dv[s:e] += gv
    return dq, dk, dv


# ----------------------------------------------------------------------------------
# Branch 2: block compression phi and compressed attention (Eq. 5).
# ----------------------------------------------------------------------------------
def gelu(x):
    """Exact GELU, x * Phi(x)."""
    return 0.5 * x * (1.0 + erf(x / math.sqrt(2.0)))


def gelu_grad(x):
    return 0.5 * (1.0 + erf(x / math.sqrt(2.0))) + x * np.exp(-0.5 * x * x) / math.sqrt(2.0 * math.pi)


def block_rows(x, valid, l):
    """Token-major flatten of each length-l block, dummy rows zeroed: [N/l, l*d]."""
    n, d = x.shape
    xz = np.where(valid[:, None], x, 0.0)
    return xz.reshape(n // l, l * d)


def pool_blocks(x, valid, l, pool, phi):
    """phi (an MLP, or the mean) of each length-l block of x: [N/l, d] and a cache."""
    flat = block_rows(x, valid, l)
    if pool == "mean":
        d = x.shape[1]
        return flat.reshape(-1, l, d).sum(axis=1) / l, {"flat": flat}
    pre = flat @ phi["w1"] + phi["b1"]
    hid = gelu(pre)
    out = hid @ phi["w2"] + phi["b2"]
    return out, {"flat": flat, "pre": pre, "hid": hid}


def pool_blocks_backward(dout, cache, valid, l, pool, phi):
    """Given d(pooled tokens), return (d tokens [N, d], dict of weight grads)."""
    d = dout.shape[1]
    if pool == "mean":
        dflat = np.repeat(dout / l, l, axis=0)
        return np.where(valid[:, None], dflat, 0.0), {}
    grads = {
        "w2": cache["hid"].T @ dout,
        "b2": dout.sum(axis=0),
    }
    dpre = (dout @ phi["w2"].T) * gelu_grad(cache["pre"])
    grads["w1"] = cache["flat"].T @ dpre
    grads["b1"] = dpre.sum(axis=0)
    # magnitude of the summed terms of each weight gradient (error scale of a sum)
    grads["abs"] = {"w2": np.abs(cache["hid"]).T @ np.abs(dout), "b2": np.abs(dout).sum(axis=0),
                    "w1": np.abs(cache["flat"]).T @ np.abs(dpre), "b1": np.abs(dpre).sum(axis=0)}
    dx = (dpre @ phi["w1"].T).reshape(-1, d)
    return np.where(valid[:, None], dx, 0.0), grads


def compress(x, valid, phi, P: Params):
    """Compressed tokens [N/l, d] of Eq. 5 and the cache needed for the backward pass."""
    return pool_blocks(x, valid, P.cmp_block, P.kv_pool, phi)


def compress_backward(dout, cache, valid, phi, P: Params):
    """Given d(compressed tokens), return (d tokens [N, d], dict of weight grads)."""
    return pool_blocks_backward(dout, cache, valid, P.cmp_block, P.kv_pool, phi)


def coarse_queries(q, valid, phi_q, P: Params):
    """Coarse queries [N/g, d]: the pooled query of Eq. 11 (q_coarsen "mean": the group's
    real queries summed and divided by g) or phi_q of each block of l = g queries, dummy
    rows zero (Eq. 13)."""
    return pool_blocks(q, valid, P.group, P.q_coarsen, phi_q)


def coarse_queries_backward(dqc, cache, valid, phi_q, P: Params):
    return pool_blocks_backward(dqc, cache, valid, P.group, P.q_coarsen, phi_q)


def block_valid(valid, l):
    return valid.reshape(-1, l).any(axis=1)


def compression_branch(q, kc, vc, cvalid, valid, P: Params, rows=None):
    n, d = q.shape
    o = np.zeros((n, d))
    lse = np.full(n, NEG_INF)
    rows = np.nonzero(valid)[0] if rows is None else rows[valid[rows]]
    for s in range(0, rows.size, 4096):
        r = rows[s:s + 4096]
        o[r], lse[r] = attend(q[r], kc, vc, cvalid, P.sm_scale(d))
    return o, lse


def compression_branch_backward(q, kc, vc, cvalid, valid, P: Params, o, lse, do):
    n, d = q.shape
    dq = np.zeros_like(q)
    dkc, dvc = np.zeros_like(kc), np.zeros_like(vc)
    rows = np.nonzero(valid)[0]
    for s in range(0, rows.size, 4096):
        r = rows[s:s + 4096]
        gq, gk, gv = attend_backward(q[r], kc, vc, cvalid, P.sm_scale(d), o[r], lse[r], do[r])
        dq[r] = gq
        dkc += gk
        dvc += gv
    return dq, dkc, dvc


def group_compression_branch(qc, kc, vc, cvalid, valid, P: Params):
    """Eq. 15: attention of the valid coarse queries to the compressed tokens, each result
    copied to the real queries of its block. Returns (o [N, d], lse [N], oc, lsec)."""
    l = P.cmp_block
    n = valid.shape[0]
    d = qc.shape[1]
    oc = np.zeros((n // l, d))
    lsec = np.full(n // l, NEG_INF)
    rows = np.nonzero(cvalid)[0]
    oc[rows], lsec[rows] = attend(qc[rows], kc, vc, cvalid, P.sm_scale(d))
    blk = np.arange(n) // l
    o = np.where(valid[:, None], oc[blk], 0.0)
    lse = np.where(valid, lsec[blk], NEG_INF)
    return o, lse, oc, lsec


def group_compression_branch_backward(qc, kc, vc, cvalid, valid, P: Params, oc, lsec, do):
    """Gradients of Eq. 15 given the branch's upstream gradient do [N, d]: the copy's
    adjoint sums do over the real queries of each block. Returns (dqc, dkc, dvc)."""
    l = P.cmp_block
    n, d = do.shape
    doc = np.where(valid[:, None], do, 0.0).reshape(n // l, l, d).sum(axis=1)
    dqc = np.zeros_like(qc)
    rows = np.nonzero(cvalid)[0]
    gq, dkc, dvc = attend_backward(qc[rows], kc, vc, cvalid, P.sm_scale(d), oc[rows], lsec[rows],
                                   doc[rows])
    dqc[rows] = gq
    return dqc, dkc, dvc


# ----------------------------------------------------------------------------------
# Branch 3: group-shared block selection (Eq. 6, 7, 10-12) and selection attention (Eq. 8).
# ----------------------------------------------------------------------------------
def group_block_scores(q, kc, valid, P: Params, groups=None, qc=None):
    """Scores [N/g, N/l'] of every selection block for every query group (or only for the
    listed groups, in that order).

    Pooled query q_p = (1/g) * sum of the group's real queries (Eq. 11), or the given
    coarse queries qc [N/g, d] (Eq. 13); compressed-block score S_pc = <q_p, kc_c> (Eq. 6,
    12, 14); a selection block of r = l'/l compressed blocks scores the mean of their
    scores. Own-ball and all-dummy blocks score -inf.
    """
    n, d = q.shape
    g, l, ls, m = P.group, P.cmp_block, P.slc_block, P.ball
    r = ls // l
    groups = np.arange(n // g) if groups is None else np.asarray(groups)
    if qc is None:
        qz = np.where(valid[:, None], q, 0.0).reshape(n // g, g, d)[groups]
        qp = qz.sum(axis=1) / g
    else:
        qp = qc[groups]
    s_cmp = qp @ kc.T                                  # [groups, N/l]
    s_blk = s_cmp.reshape(len(groups), n // ls, r).mean(axis=2)
    blk_ok = block_valid(valid, ls)
    s_blk[:, ~blk_ok] = NEG_INF
    if P.mask_own_ball:
        grp_ball = (groups * g) // m
        blk_ball = (np.arange(n // ls) * ls) // m
        s_blk[grp_ball[:, None] == blk_ball[None, :]] = NEG_INF
    return s_blk


def topk_blocks(scores, k):
    """Per row: the k highest finite scores (ties to the lower index), ascending, -1 pad."""
    rows, nb = scores.shape
    out = np.full((rows, k), -1, dtype=np.int64)
    idx = np.arange(nb)
    for p in range(rows):
        order = np.lexsort((idx, -scores[p]))
        chosen = [j for j in order[:k] if np.isfinite(scores[p, j])]
        chosen.sort()
        out[p, :len(chosen)] = chosen
    return out


def selection_keys(sel_row, valid, P: Params):
    """Token slots of the selected blocks (Eq. 8 concatenation) and their validity."""
    ls = P.slc_block
    blocks = [j for j in sel_row if j >= 0]
    slots = np.concatenate([np.arange(j * ls, (j + 1) * ls) for j in blocks]) if blocks \
        else np.zeros(0, dtype=np.int64)
    return slots, valid[slots]


def selection_branch(q, k, v, valid, sel, P: Params, groups=None):
    """Selection attention given the selected blocks sel [N/g, k*] of every group."""
    n, d = q.shape
    g = P.group
    o = np.zeros((n, d))
    lse = np.full(n, NEG_INF)
    groups = range(n // g) if groups is None else groups
    for p in groups:
        slots, kvalid = selection_keys(sel[p], valid, P)
        rows = np.nonzero(valid[p * g:(p + 1) * g])[0] + p * g
        if slots.size:
            o[rows], lse[rows] = attend(q[rows], k[slots], v[slots], kvalid, P.sm_scale(d))
    return o, lse


def selection_branch_backward(q, k, v, valid, sel, P: Params, o, lse, do):
    n, d = q.shape
    g = P.group
    dq, dk, dv = np.zeros_like(q), np.zeros_like(k), np.zeros_like(v)
    for p in range(n // g):
        slots, kvalid = selection_keys(sel[p], valid, P)
        rows = np.nonzero(valid[p * g:(p + 1) * g])[0] + p * g
        if slots.size == 0 or rows.size == 0:
            continue
        gq, gk, gv = attend_backward(q[rows], k[slots], v[slots], kvalid, P.sm_scale(d),
                                     o[rows], lse[rows], do[rows])
        dq[rows] = gq
        np.add.at(dk, slots, gk)
        np.add.at(dv, slots, gv)
    return dq, dk, dv


# ----------------------------------------------------------------------------------
# Gate (Eq. 9) and the whole layer.
# ----------------------------------------------------------------------------------
def sigmoid(x):
    return 1.0 / (1.0 + np.exp(-x))


def _f64(x):
    return np.asarray(x, dtype=np.float64)


def _phi64(phi):
    return {k: _f64(v) for k, v in phi.items()} if phi is not None else None


def forward(q, k, v, valid, gate, phi_k, phi_v, P: Params, phi_q=None):
    """Full forward pass. Arrays as described in the module docstring; phi_q is the query
    MLP of Eq. 13 (q_coarsen "mlp").

    Returns a dict with o [B,H,N,d], o_branch [3,B,H,N,d], lse [3,B,H,N], sel [B,H,N/g,k*],
    kc/vc [B,H,N/l,d], qc [B,H,N/g,d] (coarse queries), and the caches for the backward.
    """
    q, k, v, gate = _f64(q), _f64(k), _f64(v), _f64(gate)
    phi_k, phi_v, phi_q = _phi64(phi_k), _phi64(phi_v), _phi64(phi_q)
    valid = np.asarray(valid, dtype=bool)
    B, H, n, d = q.shape
    l, g = P.cmp_block, P.group
    ob = np.zeros((3, B, H, n, d))
    lse = np.full((3, B, H, n), NEG_INF)
    sel = np.full((B, H, n // g, P.topk), -1, dtype=np.int64)
    kc = np.zeros((B, H, n // l, d))
    vc = np.zeros((B, H, n // l, d))
    qc = np.zeros((B, H, n // g, d))
    ocs, lsecs = {}, {}
    caches = {}
    for b in range(B):
        vb = valid[b]
        cvalid = block_valid(vb, l)
        for h in range(H):
            qq, kk, vv = q[b, h], k[b, h], v[b, h]
            ob[0, b, h], lse[0, b, h] = ball_branch(qq, kk, vv, vb, P)
            kc[b, h], ck = compress(kk, vb, phi_k, P)
            vc[b, h], cv = compress(vv, vb, phi_v, P)
            qc[b, h], cq = coarse_queries(qq, vb, phi_q, P)
            caches[(b, h)] = (ck, cv, cq)
            if P.group_compression:
                ob[1, b, h], lse[1, b, h], ocs[(b, h)], lsecs[(b, h)] = group_compression_branch(
                    qc[b, h], kc[b, h], vc[b, h], cvalid, vb, P)
            else:
                ob[1, b, h], lse[1, b, h] = compression_branch(qq, kc[b, h], vc[b, h], cvalid, vb, P)
            sel[b, h] = topk_blocks(group_block_scores(qq, kc[b, h], vb, P, qc=qc[b, h]), P.topk)
            ob[2, b, h], lse[2, b, h] = selection_branch(qq, kk, vv, vb, sel[b, h], P)
    sg = sigmoid(gate)                                # [B, N, 3]
    o = np.zeros((B, H, n, d))
    for br in range(3):
        o += sg[:, None, :, br, None] * ob[br]
    return {"o": o, "o_branch": ob, "lse": lse, "sel": sel, "kc": kc, "vc": vc, "qc": qc,
            "oc": ocs, "lsec": lsecs, "caches": caches}


def backward(q, k, v, valid, gate, phi_k, phi_v, P: Params, fwd, do, phi_q=None):
    """Gradients of sum(o * do) with respect to q, k, v, the gate logits and the MLPs.

    The top-k selection is piecewise constant, so no gradient flows through the scores;
    phi_q therefore receives a gradient only through group compression (Eq. 15).
    Weight gradients are summed over batch, heads and blocks.
    """
    q, k, v, gate, do = _f64(q), _f64(k), _f64(v), _f64(gate), _f64(do)
    phi_k, phi_v, phi_q = _phi64(phi_k), _phi64(phi_v), _phi64(phi_q)
    valid = np.asarray(valid, dtype=bool)
    B, H, n, d = q.shape
    l = P.cmp_block
    ob, lse, sel = fwd["o_branch"], fwd["lse"], fwd["sel"]
    sg = sigmoid(gate)
    dgate = np.zeros((B, n, 3))
    dgate_abs = np.zeros((B, n, 3))
    dsg = sg * sigmoid(-gate)            # sigmoid'(x) = s(x) s(-x), no cancellation when saturated
    for br in range(3):
        dgate[:, :, br] = dsg[:, :, br] * np.sum(do * ob[br], axis=(1, 3))
        dgate_abs[:, :, br] = dsg[:, :, br] * np.sum(np.abs(do * ob[br]), axis=(1, 3))
    dq, dk, dv = np.zeros_like(q), np.zeros_like(k), np.zeros_like(v)
    wkeys = ("w1", "b1", "w2", "b2")
    dphi_k = {w: np.zeros_like(phi_k[w]) for w in wkeys} if P.kv_pool == "mlp" else {}
    dphi_v = {w: np.zeros_like(phi_v[w]) for w in wkeys} if P.kv_pool == "mlp" else {}
    abs_k = {w: np.zeros_like(phi_k[w]) for w in wkeys} if P.kv_pool == "mlp" else {}
    abs_v = {w: np.zeros_like(phi_v[w]) for w in wkeys} if P.kv_pool == "mlp" else {}
    q_mlp = P.group_compression and P.q_coarsen == "mlp"
    dphi_q = {w: np.zeros_like(phi_q[w]) for w in wkeys} if q_mlp else {}
    abs_q = {w: np.zeros_like(phi_q[w]) for w in wkeys} if q_mlp else {}
    for b in range(B):
        vb = valid[b]
        cvalid = block_valid(vb, l)
        for h in range(H):
            qq, kk, vv = q[b, h], k[b, h], v[b, h]
            dob = [sg[b, :, br, None] * do[b, h] for br in range(3)]
            g0 = ball_branch_backward(qq, kk, vv, vb, P, ob[0, b, h], lse[0, b, h], dob[0])
            ck, cv, cq = fwd["caches"][(b, h)]
            if P.group_compression:
                gqc, gkc, gvc = group_compression_branch_backward(
                    fwd["qc"][b, h], fwd["kc"][b, h], fwd["vc"][b, h], cvalid, vb, P, fwd["oc"][(b, h)],
                    fwd["lsec"][(b, h)], dob[1])
                gq, wq = coarse_queries_backward(gqc, cq, vb, phi_q, P)
                for w in wkeys if wq else ():
                    dphi_q[w] += wq[w]
                    abs_q[w] += wq["abs"][w]
            else:
                gq, gkc, gvc = compression_branch_backward(qq, fwd["kc"][b, h], fwd["vc"][b, h], cvalid,
                                                           vb, P, ob[1, b, h], lse[1, b, h], dob[1])
            dk_c, wk = compress_backward(gkc, ck, vb, phi_k, P)
            dv_c, wv = compress_backward(gvc, cv, vb, phi_v, P)
            g2 = selection_branch_backward(qq, kk, vv, vb, sel[b, h], P, ob[2, b, h], lse[2, b, h],
                                           dob[2])
            dq[b, h] = g0[0] + gq + g2[0]
            dk[b, h] = g0[1] + dk_c + g2[1]
            dv[b, h] = g0[2] + dv_c + g2[2]
            for w in wkeys if wk else ():
                dphi_k[w] += wk[w]
                dphi_v[w] += wv[w]
                abs_k[w] += wk["abs"][w]
                abs_v[w] += wv["abs"][w]
    return {"dq": dq, "dk": dk, "dv": dv, "dgate": dgate, "dphi_k": dphi_k, "dphi_v": dphi_v,
            "dphi_q": dphi_q, "abs": {"dgate": dgate_abs, "dphi_k": abs_k, "dphi_v": abs_v, "dphi_q": abs_q}}
